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

// bf16 of the exact sum a + b, round to nearest even.  The float32 sum s and
// its rounding error e are exact (TwoSum); rounding s again to bf16 can only
// differ from rounding a + b once when s is a bf16 tie (low half 0x8000), and
// there the sign of e decides: the exact sum is farther from zero than s when
// e has s's sign (round the magnitude up), else nearer (truncate).
__device__ __forceinline__ uint16_t sum_to_bf16(float a, float b) {
  const float s = a + b;
  const uint32_t u = __float_as_uint(s);
  if ((u & 0xFFFFu) != 0x8000u || (u & 0x7F800000u) == 0x7F800000u) return f32_to_bf16(s);
  const float bb = s - a;
  const float e = (a - (s - bb)) + (b - bb);
  if (e == 0.f) return f32_to_bf16(s);
  return (uint16_t)((u >> 16) + (((e > 0.f) == (s > 0.f)) ? 1u : 0u));
}

template <typename T>
struct Elem;
template <>
struct Elem<bf16_t> {
  static constexpr int kBytes = 2;
  __device__ static float to_f32(const void* base, size_t i) { return bf16_to_f32(((const uint16_t*)base)[i]); }
  __device__ static void store(void* base, size_t i, float v) { ((uint16_t*)base)[i] = f32_to_bf16(v); }
  // round(a + b) of the exact sum
  __device__ static void store_sum(void* base, size_t i, float a, float b) { ((uint16_t*)base)[i] = sum_to_bf16(a, b); }
};
template <>
struct Elem<float> {
  static constexpr int kBytes = 4;
  __device__ static float to_f32(const void* base, size_t i) { return ((const float*)base)[i]; }
  __device__ static void store(void* base, size_t i, float v) { ((float*)base)[i] = v; }
  __device__ static void store_sum(void* base, size_t i, float a, float b) { ((float*)base)[i] = a + b; }
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

// Top-K candidates as 64-bit keys: the high word is the float's bits mapped to
// an order-preserving unsigned integer, the low word is the inverted token id,
// so a larger key is a larger value, or an equal value with a smaller id.
// Key 0 is below every real candidate and marks an empty slot.
__device__ __forceinline__ uint32_t ord_f32(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key_value(uint64_t k) {
  const uint32_t u = (uint32_t)(k >> 32);
  return __uint_as_float((u & 0x80000000u) ? (u & 0x7FFFFFFFu) : ~u);
}
__device__ __forceinline__ int key_id(uint64_t k) { return (int)(~(uint32_t)k); }
__device__ __forceinline__ uint64_t make_key(float v, int id) {
  v = v == 0.f ? 0.f : v;  // -0 and +0 are one value (ties go by id)
  return ((uint64_t)ord_f32(v) << 32) | (uint32_t)(~(uint32_t)id);
}

// Exact top-K of two descending key lists: the element-wise maxima of a[i] and
// b[K-1-i] are the top K of the union and form a bitonic sequence, which
// log2(K) compare-exchange stages sort (bitonic merge).  K is 4, 8 or 16.
template <int K>
__device__ __forceinline__ void merge_topk(uint64_t (&a)[K], const uint64_t (&b)[K]) {
#pragma unroll
  for (int i = 0; i < K; ++i) a[i] = b[K - 1 - i] > a[i] ? b[K - 1 - i] : a[i];
#pragma unroll
  for (int st = K / 2; st >= 1; st >>= 1) {
#pragma unroll
    for (int i = 0; i < K; ++i) {
      if ((i & st) == 0) {
        const int j = i + st;
        const bool sw = a[j] > a[i];
        const uint64_t x = a[i], y = a[j];
        a[i] = sw ? y : x;
        a[j] = sw ? x : y;
      }
    }
  }
}

// Online softmax statistics of a set of logits: max m, smallest argmax,
// S = sum e^(z-m), T = sum e^(z-m) (z-m).  merge() combines two disjoint sets
// without branches; an empty set has m = -inf.
struct RowStats {
  float m, S, T;
  int am;
  __device__ __forceinline__ void init() {
    m = -__builtin_huge_valf();
    S = 0.f;
    T = 0.f;
    am = 0x7FFFFFFF;
  }
  __device__ __forceinline__ void merge(float m2, float S2, float T2, int am2) {
    const float M = fmaxf(m, m2);
    const bool z1 = m == -__builtin_huge_valf(), z2 = m2 == -__builtin_huge_valf();
    const float d1 = z1 ? 0.f : m - M, d2 = z2 ? 0.f : m2 - M;
    const float e1 = z1 ? 0.f : __expf(d1), e2 = z2 ? 0.f : __expf(d2);
    T = e1 * (T + d1 * S) + e2 * (T2 + d2 * S2);
    S = e1 * S + e2 * S2;
    am = m > m2 ? am : (m2 > m ? am2 : min(am, am2));
    m = M;
  }
  template <int LEVEL>
  __device__ __forceinline__ void merge_level();
};

// Butterfly partner exchange at level 0..5 of a wave (all 64 lanes active):
// levels 0-3 pair lanes inside a 16-lane row with DPP moves (xor 1, xor 2,
// mirror within 8, mirror within 16); levels 4 and 5 pair rows (xor 16, xor 32)
// with gfx950's v_permlane16_swap / v_permlane32_swap.  Swapping a register
// with itself leaves, in the two results, each lane's own value and its
// partner row's value; the lane picks the partner's.
// After levels 0..L every lane holds the combination of its 2^(L+1) lanes.
template <int LEVEL>
__device__ __forceinline__ int xchg(int v) {
  if constexpr (LEVEL == 0) return __builtin_amdgcn_mov_dpp(v, 0xB1, 0xF, 0xF, false);   // quad_perm 1,0,3,2
  if constexpr (LEVEL == 1) return __builtin_amdgcn_mov_dpp(v, 0x4E, 0xF, 0xF, false);   // quad_perm 2,3,0,1
  if constexpr (LEVEL == 2) return __builtin_amdgcn_mov_dpp(v, 0x141, 0xF, 0xF, false);  // row_half_mirror
  if constexpr (LEVEL == 3) return __builtin_amdgcn_mov_dpp(v, 0x140, 0xF, 0xF, false);  // row_mirror
  const int lane = (int)(threadIdx.x & 63);
  if constexpr (LEVEL == 4) {
    const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);  // odd rows <-> even rows
    return (lane & 16) ? (int)r[0] : (int)r[1];
  }
  const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);    // upper half <-> lower half
  return (lane & 32) ? (int)r[0] : (int)r[1];
}
template <int LEVEL>
__device__ __forceinline__ float xchg(float v) {
  return __int_as_float(xchg<LEVEL>(__float_as_int(v)));
}
template <int LEVEL>
__device__ __forceinline__ uint64_t xchg(uint64_t v) {
  const uint32_t lo = (uint32_t)xchg<LEVEL>((int)(uint32_t)v), hi = (uint32_t)xchg<LEVEL>((int)(uint32_t)(v >> 32));
  return ((uint64_t)hi << 32) | lo;
}

template <int LEVEL>
__device__ __forceinline__ void RowStats::merge_level() {
  const float m2 = xchg<LEVEL>(m), S2 = xchg<LEVEL>(S), T2 = xchg<LEVEL>(T);
  const int am2 = xchg<LEVEL>(am);
  merge(m2, S2, T2, am2);
}

// Exchange a sorted top-K key list with the butterfly partner and keep the merged top K.
template <int K, int LEVEL>
__device__ __forceinline__ void merge_topk_level(uint64_t (&k)[K]) {
  uint64_t p[K];
#pragma unroll
  for (int i = 0; i < K; ++i) p[i] = xchg<LEVEL>(k[i]);
  merge_topk<K>(k, p);
}


// Cross-workgroup hand-off through global memory on a multi-XCD GPU.
// Each XCD has its own L2, so data that one workgroup hands to another inside
// a kernel is written and read with device-coherent (agent-scope) accesses,
// which the hardware performs at the device coherence point (sc1 bit):
//   producer: st_dev*(...) for the data, then stores_done() before the
//             workgroup takes its ticket with a device-scope atomic;
//   consumer: ld_dev*(...) for the data after winning the ticket.
// No L2 write-back or invalidate is needed (a __threadfence() on every wave
// would write back and invalidate the whole L2 under every other workgroup).
// A location is written by at most one workgroup per step.
__device__ __forceinline__ void st_dev(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_dev(int32_t* p, int32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_dev4(float* p, f32x4 v) {  // p 16-byte aligned
  unsigned long long* q = reinterpret_cast<unsigned long long*>(p);
  const unsigned long long lo = ((unsigned long long)__float_as_uint(v.y) << 32) | __float_as_uint(v.x);
  const unsigned long long hi = ((unsigned long long)__float_as_uint(v.w) << 32) | __float_as_uint(v.z);
  __hip_atomic_store(q, lo, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(q + 1, hi, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_dev(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int32_t ld_dev(const int32_t* p) {
  return __hip_atomic_load(const_cast<int32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ f32x4 ld_dev4(const float* p) {
  unsigned long long* q = reinterpret_cast<unsigned long long*>(const_cast<float*>(p));
  const unsigned long long lo = __hip_atomic_load(q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const unsigned long long hi = __hip_atomic_load(q + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return f32x4{__uint_as_float((uint32_t)lo), __uint_as_float((uint32_t)(lo >> 32)), __uint_as_float((uint32_t)hi),
               __uint_as_float((uint32_t)(hi >> 32))};
}
// Wait until this wave's memory operations have completed (stores acknowledged).
// The signal fences keep the compiler from moving memory operations across the
// wait (they emit no instruction).
__device__ __forceinline__ void stores_done() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// Completion ticket: an agent-scope release read-modify-write.  Every store of
// this workgroup that happens before it (this wave's own, and the other waves'
// through the workgroup barrier before it) is ordered before the new count, and
// the counter's read-modify-writes form one release sequence, so the workgroup
// that reads the final count and then takes acquire_agent() sees all of them.
__device__ __forceinline__ int32_t ticket_release(int32_t* p) {
  return __hip_atomic_fetch_add(p, 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void acquire_agent() { __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent"); }

// Intra-wave ordering point for LDS data written and read by the same wave.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

}  // namespace respec
