// LM head: logits z[m][v] = sum_c x[m][c] * W[v][c]  (W row-major [V][Hd]).
//
// The target distribution of every tree node, P_t = softmax(z) (ReSpec,
// Section 3.2.1), starts here.  The M dimension is the number of draft nodes
// (tens to a few hundred), so the GEMM is skinny: W (hundreds of MB) is
// streamed from HBM exactly once and is the roofline.
//
// Tiling: a workgroup owns 128 vocabulary rows (4 waves x 32) and one tile of
// 16*MB token rows.  The contraction runs on the matrix cores with W as the A
// operand (16-byte fragments loaded straight from HBM, next K-chunk prefetched
// into registers) and x as the B operand (staged per 512-byte K-chunk in LDS,
// rows padded by 16 bytes against bank conflicts).  Output lane layout gives
// each lane 4 consecutive vocabulary entries of one token row: 16-byte stores.
#include "common.hpp"
#include "kernels.hpp"

namespace respec {

constexpr int kLmChunkBytes = 512;                  // bytes of a row per K step
constexpr int kLmPieces = kLmChunkBytes / 64;       // mma_k64 calls per K step
constexpr int kLmXStride = kLmChunkBytes + 16;      // LDS row stride of the x tile

template <typename T, int MB>
__global__ __launch_bounds__(256) void lmhead_kernel(LmArgs a) {
  constexpr int ES = Elem<T>::kBytes;
  __shared__ __align__(16) unsigned char sx[16 * MB * kLmXStride];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int vw = blockIdx.x * 128 + 32 * wave;  // first vocabulary row of this wave
  const int m0 = blockIdx.y * 16 * MB;
  const size_t row_bytes = (size_t)a.hidden_size * ES;
  const int n_steps = (int)(row_bytes / kLmChunkBytes);

  const char* wrow[2];
  bool wok[2];
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    const int v = vw + 16 * nb + lr;
    wok[nb] = v < a.vocab;
    wrow[nb] = reinterpret_cast<const char*>(a.w) + (size_t)(wok[nb] ? v : 0) * row_bytes + lg * 16;
  }
  const char* xbase = reinterpret_cast<const char*>(a.x);

  f32x4 acc[2][MB];
#pragma unroll
  for (int nb = 0; nb < 2; ++nb)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[nb][mb] = f32x4{0.f, 0.f, 0.f, 0.f};

  u32x4 wc[2][kLmPieces];
#pragma unroll
  for (int nb = 0; nb < 2; ++nb)
#pragma unroll
    for (int kp = 0; kp < kLmPieces; ++kp)
      wc[nb][kp] = wok[nb] ? ld16(wrow[nb] + kp * 64) : u32x4{0, 0, 0, 0};

  for (int step = 0; step < n_steps; ++step) {
    // prefetch the next K step of W
    u32x4 wn[2][kLmPieces];
    const bool more = step + 1 < n_steps;
    const size_t next_off = (size_t)(step + 1) * kLmChunkBytes;
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int kp = 0; kp < kLmPieces; ++kp)
        wn[nb][kp] = (more && wok[nb]) ? ld16(wrow[nb] + next_off + kp * 64) : u32x4{0, 0, 0, 0};

    // stage x[m0 .. m0+16*MB)[step chunk] into LDS
    __syncthreads();
    for (int idx = threadIdx.x; idx < 16 * MB * (kLmChunkBytes / 16); idx += blockDim.x) {
      const int r = idx / (kLmChunkBytes / 16), pc = idx % (kLmChunkBytes / 16);
      const int m = m0 + r;
      const u32x4 v = m < a.m_rows ? ld16(xbase + (size_t)m * row_bytes + (size_t)step * kLmChunkBytes + pc * 16)
                                   : u32x4{0, 0, 0, 0};
      *reinterpret_cast<u32x4*>(sx + r * kLmXStride + pc * 16) = v;
    }
    __syncthreads();

#pragma unroll
    for (int kp = 0; kp < kLmPieces; ++kp) {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const u32x4 xb = *reinterpret_cast<const u32x4*>(sx + (16 * mb + lr) * kLmXStride + kp * 64 + lg * 16);
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) acc[nb][mb] = mma_k64(T{}, wc[nb][kp], xb, acc[nb][mb]);
      }
    }
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int kp = 0; kp < kLmPieces; ++kp) wc[nb][kp] = wn[nb][kp];
  }

  // lane holds z[m0 + 16*mb + lr][vw + 16*nb + 4*lg + i]
  const bool vec_ok = (a.vocab & 3) == 0;
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const int m = m0 + 16 * mb + lr;
      const int v = vw + 16 * nb + 4 * lg;
      if (m >= a.m_rows) continue;
      float* dst = a.logits + (size_t)m * a.vocab + v;
      if (vec_ok && v + 3 < a.vocab) {
        *reinterpret_cast<f32x4*>(dst) = acc[nb][mb];
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (v + i < a.vocab) dst[i] = acc[nb][mb][i];
      }
    }
  }
}

template <typename T>
static hipError_t launch_mb(int mb, dim3 grid, const LmArgs& a, hipStream_t s) {
  switch (mb) {
    case 1: hipLaunchKernelGGL((lmhead_kernel<T, 1>), grid, dim3(256), 0, s, a); break;
    case 2: hipLaunchKernelGGL((lmhead_kernel<T, 2>), grid, dim3(256), 0, s, a); break;
    case 3: hipLaunchKernelGGL((lmhead_kernel<T, 3>), grid, dim3(256), 0, s, a); break;
    case 4: hipLaunchKernelGGL((lmhead_kernel<T, 4>), grid, dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_lmhead(int dtype, int mb, dim3 grid, const LmArgs& a, hipStream_t s) {
  return dtype == 1 ? launch_mb<bf16_t>(mb, grid, a, s) : launch_mb<float>(mb, grid, a, s);
}

}  // namespace respec
