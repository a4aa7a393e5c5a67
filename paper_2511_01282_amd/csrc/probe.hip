// Measurement probes: a plain streaming read and a matrix-core loop, the two
// ceilings the verification kernels are reported against beside the vendor
// peaks.  See include/respec_probe.h.
#include "../../include/respec_probe.h"
#include "common.hpp"

namespace respec {
namespace {

constexpr size_t kStep = 256 * 16;  // bytes a workgroup reads per step

template <int DEPTH>
__global__ __launch_bounds__(256) void probe_read_kernel(const char* buf, size_t chunk, uint32_t* sink) {
  const char* p = buf + (size_t)blockIdx.x * chunk + threadIdx.x * 16;
  const size_t steps = chunk / kStep;
  uint32_t acc = 0;
  size_t s = 0;
  for (; s + DEPTH <= steps; s += DEPTH) {
    u32x4 v[DEPTH];
#pragma unroll
    for (int u = 0; u < DEPTH; ++u) v[u] = ld16(p + (s + u) * kStep);
#pragma unroll
    for (int u = 0; u < DEPTH; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (; s < steps; ++s) {
    const u32x4 v = ld16(p + s * kStep);
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
  for (int o = 32; o > 0; o >>= 1) acc ^= (uint32_t)__shfl_xor((int)acc, o, 64);
  __shared__ uint32_t sh[4];
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) sink[blockIdx.x] = sh[0] ^ sh[1] ^ sh[2] ^ sh[3];
}

// Eight independent accumulation chains per wave, issued back to back.  The
// instructions are inline assembly with the accumulators updated in place:
// written as builtins, the compiler rotates the chains through other registers
// every iteration (several VALU copies per product), which measures the copies.
template <int SHAPE>
__global__ __launch_bounds__(256) void probe_mfma_kernel(int iters, float* sink) {
  // operands from the thread index (not known at compile time)
  typedef float f32x16 __attribute__((ext_vector_type(16)));
  const uint32_t t = threadIdx.x + 1;
  const u32x4 a = {t * 0x3F800000u & 0x3F803F80u, 0x3F803F80u, t & 0x00FF00FFu, 0x3C003C00u};
  const u32x4 b = {0x3C003C00u, t << 4, 0x3F803F80u, t * 7u & 0x00FF00FFu};
  float total = 0.f;
  if constexpr (SHAPE == 0) {
    f32x4 c[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) c[k] = f32x4{(float)k, 0.f, 0.f, 0.f};  // distinct chains
    for (int it = 0; it < iters; ++it) {
#pragma unroll
      for (int k = 0; k < 8; ++k) asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(c[k]) : "v"(a), "v"(b));
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) total += c[k].x + c[k].y + c[k].z + c[k].w;
  } else {
    f32x16 c[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      c[k] = f32x16{};
      c[k][0] = (float)k;
    }
    for (int it = 0; it < iters; ++it) {
#pragma unroll
      for (int k = 0; k < 8; ++k) asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(c[k]) : "v"(a), "v"(b));
    }
#pragma unroll
    for (int k = 0; k < 8; ++k)
#pragma unroll
      for (int e = 0; e < 16; ++e) total += c[k][e];
  }
  sink[(size_t)blockIdx.x * 256 + threadIdx.x] = total;
}

}  // namespace
}  // namespace respec

extern "C" {

int respec_probe_read(const void* buf, size_t bytes, int32_t workgroups, int32_t depth, uint32_t* sink,
                      void* stream) {
  if (!buf || !sink || workgroups < 1 || workgroups > 65536 || ((uintptr_t)buf % 16) != 0 ||
      bytes % (respec::kStep * (size_t)workgroups) != 0)
    return 1;
  const size_t chunk = bytes / (size_t)workgroups;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const char* p = static_cast<const char*>(buf);
  switch (depth) {
    case 4: hipLaunchKernelGGL(respec::probe_read_kernel<4>, dim3(workgroups), dim3(256), 0, s, p, chunk, sink); break;
    case 8: hipLaunchKernelGGL(respec::probe_read_kernel<8>, dim3(workgroups), dim3(256), 0, s, p, chunk, sink); break;
    case 16: hipLaunchKernelGGL(respec::probe_read_kernel<16>, dim3(workgroups), dim3(256), 0, s, p, chunk, sink); break;
    default: return 1;
  }
  return hipGetLastError() == hipSuccess ? 0 : 2;
}

int respec_probe_mfma(int32_t workgroups, int32_t iters, int32_t shape, float* sink, void* stream) {
  if (!sink || workgroups < 1 || iters < 1 || (shape != 0 && shape != 1)) return 1;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (shape == 0)
    hipLaunchKernelGGL(respec::probe_mfma_kernel<0>, dim3(workgroups), dim3(256), 0, s, iters, sink);
  else
    hipLaunchKernelGGL(respec::probe_mfma_kernel<1>, dim3(workgroups), dim3(256), 0, s, iters, sink);
  return hipGetLastError() == hipSuccess ? 0 : 2;
}

}  // extern "C"
