// LM head: logits z[m][v] = sum_c x[m][c] * W[v][c]  (W row-major [V][Hd]).
//
// The target distribution of every tree node, P_t = softmax(z) (ReSpec,
// Section 3.2.1), starts here.  The M dimension is the number of draft nodes
// (tens to a few hundred), so the GEMM is skinny: W (hundreds of MB) is
// streamed from HBM exactly once and is the roofline.
//
// Tiling: a workgroup owns 64 vocabulary rows (4 waves x 16) and one tile of
// 16*MB token rows; about two workgroups share a CU.  The contraction runs on
// the matrix cores with W as the A operand and x as the B operand.
//   - W fragments (16 bytes per lane) go straight from HBM to registers in a
//     two-deep pipeline: while K step c is multiplied, step c+1 is in flight
//     and step c+2 is issued right after.
//   - x is staged per 512-byte K step in a double-buffered, padded LDS tile.
//     Its loads are issued before the next W loads, so waiting for them never
//     waits for W (memory counters drain in issue order).
//   - Tiles are numbered so that the M tiles of one vocabulary tile run on the
//     same XCD at the same time and share W through that XCD's L2.
// Output lane layout gives each lane 4 consecutive vocabulary entries of one
// token row: 16-byte stores.  When the full step runs, the epilogue also
// reduces each token row's 64 logits of this workgroup to a TilePartial
// (online-softmax statistics and the exact top-K), so the vocabulary pass never
// re-reads the logits.
#include "common.hpp"
#include "kernels.hpp"

namespace respec {

constexpr int kLmRows = 64;                         // vocabulary rows per workgroup
constexpr int kLmChunkBytes = 512;                  // bytes of a row per K step
constexpr int kLmPieces = kLmChunkBytes / 64;       // mma_k64 calls per K step
constexpr int kLmXStride = kLmChunkBytes + 16;      // LDS row stride of the x tile

template <int MB>
struct XStage {
  static constexpr int kPieces = 16 * MB * (kLmChunkBytes / 16);  // 16-byte pieces per tile
  static constexpr int kPerThread = (kPieces + 255) / 256;
  u32x4 v[kPerThread];
};

template <int MB>
__device__ __forceinline__ void x_load(XStage<MB>& xs, const char* xbase, size_t row_bytes, int m0, int m_rows,
                                       int step) {
#pragma unroll
  for (int t = 0; t < XStage<MB>::kPerThread; ++t) {
    const int idx = threadIdx.x + 256 * t;
    const int r = idx / (kLmChunkBytes / 16), pc = idx % (kLmChunkBytes / 16);
    const int m = m0 + r;
    xs.v[t] = (idx < XStage<MB>::kPieces && m < m_rows)
                  ? ld16(xbase + (size_t)m * row_bytes + (size_t)step * kLmChunkBytes + pc * 16)
                  : u32x4{0, 0, 0, 0};
  }
}

template <int MB>
__device__ __forceinline__ void x_store(const XStage<MB>& xs, unsigned char* sx) {
#pragma unroll
  for (int t = 0; t < XStage<MB>::kPerThread; ++t) {
    const int idx = threadIdx.x + 256 * t;
    if (idx < XStage<MB>::kPieces) {
      const int r = idx / (kLmChunkBytes / 16), pc = idx % (kLmChunkBytes / 16);
      *reinterpret_cast<u32x4*>(sx + r * kLmXStride + pc * 16) = xs.v[t];
    }
  }
}

__device__ __forceinline__ void w_load(u32x4 (&w)[kLmPieces], const char* wrow, bool ok, size_t off) {
#pragma unroll
  for (int kp = 0; kp < kLmPieces; ++kp) w[kp] = ok ? ld16(wrow + off + kp * 64) : u32x4{0, 0, 0, 0};
}

template <typename T, int MB>
__device__ __forceinline__ void mma_step(f32x4 (&acc)[MB], const u32x4 (&w)[kLmPieces], const unsigned char* sx,
                                         int lr, int lg) {
#pragma unroll
  for (int kp = 0; kp < kLmPieces; ++kp) {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const u32x4 xb = *reinterpret_cast<const u32x4*>(sx + (16 * mb + lr) * kLmXStride + kp * 64 + lg * 16);
      acc[mb] = mma_k64(T{}, w[kp], xb, acc[mb]);
    }
  }
}

// Per-row statistics of this workgroup's 64 logits of every token row, written
// as one TilePartial: lane-local statistics and sort of 4 values, bitonic
// top-K merges across the 4 lane groups of a row (shuffles), then across the 4
// waves (LDS, then DPP within a quad of lanes).
template <int MB, int KO>
__device__ __forceinline__ void tile_partials(const f32x4 (&acc)[MB], unsigned char* lds, int vw, int vt, int m0,
                                              const LmArgs& a, int lane, int wave) {
  constexpr int W = TilePartial<KO>::kWords;
  constexpr int ROWS = 16 * MB;
  const int lr = lane & 15, lg = lane >> 4;
  uint32_t* s_part = reinterpret_cast<uint32_t*>(lds);  // [4 waves][ROWS][W]
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    uint64_t key[KO];
    float mx = kNegInf;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int col = vw + 4 * lg + i;
      mx = col < a.vocab ? fmaxf(mx, acc[mb][i]) : mx;
    }
    RowStats st;
    st.init();
    st.m = mx;
#pragma unroll
    for (int i = 0; i < KO; ++i) {
      const int col = vw + 4 * lg + i;
      const bool ok = i < 4 && col < a.vocab;
      key[i] = ok ? make_key(acc[mb][i & 3], col) : 0ull;
      if (i < 4) {
        const float d = acc[mb][i] - mx;
        const float e = ok ? __expf(d) : 0.f;
        st.S += e;
        st.T += ok ? e * d : 0.f;
        st.am = (ok && acc[mb][i] == mx) ? min(st.am, col) : st.am;
      }
    }
    // sort the first 4 keys (the rest are empty)
    auto cas = [&](int x, int y) {
      const bool sw = key[y] > key[x];
      const uint64_t kx = key[x], ky = key[y];
      key[x] = sw ? ky : kx;
      key[y] = sw ? kx : ky;
    };
    cas(0, 1); cas(2, 3); cas(0, 2); cas(1, 3); cas(1, 2);
    st.merge_level<4>();  // lane groups of a row: xor 16, xor 32
    merge_topk_level<KO, 4>(key);
    st.merge_level<5>();
    merge_topk_level<KO, 5>(key);
    if (lg == 0) {
      uint32_t* dst = s_part + ((size_t)wave * ROWS + 16 * mb + lr) * W;
      dst[0] = __float_as_uint(st.m);
      dst[1] = __float_as_uint(st.S);
      dst[2] = __float_as_uint(st.T);
      dst[3] = (uint32_t)st.am;
#pragma unroll
      for (int i = 0; i < KO; ++i) {
        dst[4 + 2 * i] = (uint32_t)key[i];
        dst[5 + 2 * i] = (uint32_t)(key[i] >> 32);
      }
    }
  }
  __syncthreads();
  // across the 4 waves: the 4 lanes of a quad hold one row's 4 wave lists
  for (int t = threadIdx.x; t < 4 * ROWS; t += blockDim.x) {
    const int r = t >> 2, q = t & 3;
    const int m = m0 + r;
    if (m >= a.m_rows) continue;  // uniform over the quad
    const uint32_t* src = s_part + ((size_t)q * ROWS + r) * W;
    RowStats st;
    st.m = __uint_as_float(src[0]);
    st.S = __uint_as_float(src[1]);
    st.T = __uint_as_float(src[2]);
    st.am = (int)src[3];
    uint64_t key[KO];
#pragma unroll
    for (int i = 0; i < KO; ++i) key[i] = ((uint64_t)src[5 + 2 * i] << 32) | src[4 + 2 * i];
    st.merge_level<0>();
    merge_topk_level<KO, 0>(key);
    st.merge_level<1>();
    merge_topk_level<KO, 1>(key);
    if (q == 0) {
      u32x4* dst = reinterpret_cast<u32x4*>(a.partials + ((size_t)m * a.n_vtiles + vt) * W);
      dst[0] = u32x4{__float_as_uint(st.m), __float_as_uint(st.S), __float_as_uint(st.T), (uint32_t)st.am};
#pragma unroll
      for (int i = 0; i < KO; i += 2)
        dst[1 + i / 2] = u32x4{(uint32_t)key[i], (uint32_t)(key[i] >> 32), (uint32_t)key[i + 1],
                               (uint32_t)(key[i + 1] >> 32)};
    }
  }
}

template <typename T, int MB, int KO>
__global__ __launch_bounds__(256) void lmhead_kernel(LmArgs a) {
  constexpr int ES = Elem<T>::kBytes;
  __shared__ __align__(16) unsigned char sx[2][16 * MB * kLmXStride];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  // tile order: the M tiles of one vocabulary tile are 8 block ids apart (same XCD)
  const int n_mt = a.n_mtiles;
  const int id = blockIdx.x;
  const int grp = id / (8 * n_mt), rem = id % (8 * n_mt);
  const int vt = grp * 8 + rem % 8, mt = rem / 8;
  if (vt * kLmRows >= a.vocab) return;
  const int vw = vt * kLmRows + 16 * wave;  // first vocabulary row of this wave
  const int m0 = mt * 16 * MB;
  const size_t row_bytes = (size_t)a.hidden_size * ES;
  const int n_steps = (int)(row_bytes / kLmChunkBytes);

  // Each workgroup walks the K steps from its own starting step (wrapping
  // around): workgroups that run at the same time then read different column
  // ranges of their rows, which spreads the requests over the memory channels
  // (rows are 8 KB apart, so equal column offsets would land on the same ones).
  const int rot = vt % n_steps;
  const int v = vw + lr;
  const bool wok = v < a.vocab;
  const char* wrow = reinterpret_cast<const char*>(a.w) + (size_t)(wok ? v : 0) * row_bytes + lg * 16;
  const char* xbase = reinterpret_cast<const char*>(a.x);

  f32x4 acc[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) acc[mb] = f32x4{0.f, 0.f, 0.f, 0.f};

  u32x4 wa[kLmPieces], wb[kLmPieces];
  XStage<MB> xs;
  auto step_of = [&](int c) { return c + rot < n_steps ? c + rot : c + rot - n_steps; };
  w_load(wa, wrow, wok, (size_t)step_of(0) * kLmChunkBytes);
  if (n_steps > 1) w_load(wb, wrow, wok, (size_t)step_of(1) * kLmChunkBytes);
  x_load<MB>(xs, xbase, row_bytes, m0, a.m_rows, step_of(0));
  x_store<MB>(xs, sx[0]);
  __syncthreads();

  for (int c = 0; c < n_steps; c += 2) {
    // ---- step c: wa, sx[0] ----
    if (c + 1 < n_steps) x_load<MB>(xs, xbase, row_bytes, m0, a.m_rows, step_of(c + 1));
    mma_step<T, MB>(acc, wa, sx[0], lr, lg);
    if (c + 2 < n_steps) w_load(wa, wrow, wok, (size_t)step_of(c + 2) * kLmChunkBytes);
    if (c + 1 >= n_steps) break;
    x_store<MB>(xs, sx[1]);
    __syncthreads();
    // ---- step c+1: wb, sx[1] ----
    if (c + 2 < n_steps) x_load<MB>(xs, xbase, row_bytes, m0, a.m_rows, step_of(c + 2));
    mma_step<T, MB>(acc, wb, sx[1], lr, lg);
    if (c + 3 < n_steps) w_load(wb, wrow, wok, (size_t)step_of(c + 3) * kLmChunkBytes);
    if (c + 2 < n_steps) {
      x_store<MB>(xs, sx[0]);
      __syncthreads();
    }
  }

  // lane holds z[m0 + 16*mb + lr][vw + 4*lg + i]
  const bool vec_ok = (a.vocab & 3) == 0;
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const int m = m0 + 16 * mb + lr;
    const int vv = vw + 4 * lg;
    if (m >= a.m_rows) continue;
    float* dst = a.logits + (size_t)m * a.vocab + vv;
    if (vec_ok && vv + 3 < a.vocab) {
      *reinterpret_cast<f32x4*>(dst) = acc[mb];
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (vv + i < a.vocab) dst[i] = acc[mb][i];
    }
  }
  if (a.partials) {
    __syncthreads();  // the x tiles in LDS are no longer read
    tile_partials<MB, KO>(acc, &sx[0][0], vw, vt, m0, a, lane, wave);
  }
}

template <typename T, int KO>
static hipError_t launch_mb(int mb, dim3 grid, const LmArgs& a, hipStream_t s) {
  switch (mb) {
    case 1: hipLaunchKernelGGL((lmhead_kernel<T, 1, KO>), grid, dim3(256), 0, s, a); break;
    case 2: hipLaunchKernelGGL((lmhead_kernel<T, 2, KO>), grid, dim3(256), 0, s, a); break;
    case 3: hipLaunchKernelGGL((lmhead_kernel<T, 3, KO>), grid, dim3(256), 0, s, a); break;
    case 4: hipLaunchKernelGGL((lmhead_kernel<T, 4, KO>), grid, dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_lmhead(int dtype, int mb, int ko, const LmArgs& a, hipStream_t s) {
  const int n_vt = (a.vocab + kLmRows - 1) / kLmRows;
  const int n_grp = (n_vt + 7) / 8;
  dim3 grid(n_grp * 8 * a.n_mtiles);
  if (ko == 8) return dtype == 1 ? launch_mb<bf16_t, 8>(mb, grid, a, s) : launch_mb<float, 8>(mb, grid, a, s);
  if (ko == 16) return dtype == 1 ? launch_mb<bf16_t, 16>(mb, grid, a, s) : launch_mb<float, 16>(mb, grid, a, s);
  return hipErrorInvalidValue;
}

}  // namespace respec
