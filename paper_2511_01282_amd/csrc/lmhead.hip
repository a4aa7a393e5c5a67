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
//   - W fragments (16 bytes per lane) go straight from HBM to registers, and
//     each thread's share of the x tile with them, in a ring of two or three K
//     steps: while step c is multiplied the next ones are in flight, and the
//     requests of step c + ring are issued right after (memory counters drain
//     in issue order, so waiting for step c never waits for newer requests).
//   - x is staged per 512-byte K step in a double-buffered, padded LDS tile.
//   - Tiles are numbered so that the M tiles of one vocabulary tile run on the
//     same XCD at the same time and share W through that XCD's L2.
// Output lane layout gives each lane 4 consecutive vocabulary entries of one
// token row: 16-byte stores.  When the full step runs, the epilogue also
// reduces each token row's 64 logits of a statistics tile to its online-softmax
// statistics {max, sum, entropy sum, argmax} (kTileWords), so that the
// vocabulary pass reads them, and of the logits only the few tiles whose
// maxima can hold a row's top-K.
#include <atomic>

#include "common.hpp"
#include "kernels.hpp"

namespace respec {

constexpr int kLmRows = 64;                         // vocabulary rows per workgroup
constexpr int kLmChunkBytes = 512;                  // bytes of a row per K step
constexpr int kLmPieces = kLmChunkBytes / 64;       // mma_k64 calls per K step
constexpr int kLmXStride = kLmChunkBytes + 16;      // LDS row stride of the x tile

// x tile of one K step: 16*MB token rows x 512 bytes, in 16-byte pieces
template <int MB>
struct XStage {
  static constexpr int kPieces = 16 * MB * (kLmChunkBytes / 16);  // 16-byte pieces per tile
  static constexpr int kPerThread = (kPieces + 255) / 256;
};

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
// as one tile partial {m, S, T, argmax}: lane-local statistics of 4 values,
// merged across the 4 lane groups of a row (permlane swaps), then across the
// 4 waves (LDS, then DPP within a quad of lanes).
template <int MB>
__device__ __forceinline__ void tile_partials(const f32x4 (&acc)[MB], unsigned char* lds, int vw, int vt, int m0,
                                              const LmArgs& a, int lane, int wave) {
  constexpr int ROWS = 16 * MB;
  const int lr = lane & 15, lg = lane >> 4;
  u32x4* s_part = reinterpret_cast<u32x4*>(lds);  // [4 waves][ROWS]
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
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
    for (int i = 0; i < 4; ++i) {
      const int col = vw + 4 * lg + i;
      const bool ok = col < a.vocab;
      const float d = acc[mb][i] - mx;
      const float e = ok ? __expf(d) : 0.f;
      st.S += e;
      st.T += ok ? e * d : 0.f;
      st.am = (ok && acc[mb][i] == mx) ? min(st.am, col) : st.am;
    }
    st.merge_level<4>();  // lane groups of a row: xor 16, xor 32
    st.merge_level<5>();
    if (lg == 0)
      s_part[wave * ROWS + 16 * mb + lr] =
          u32x4{__float_as_uint(st.m), __float_as_uint(st.S), __float_as_uint(st.T), (uint32_t)st.am};
  }
  __syncthreads();
  // across the 4 waves: the 4 lanes of a quad hold one row's 4 wave statistics
  for (int t = threadIdx.x; t < 4 * ROWS; t += blockDim.x) {
    const int r = t >> 2, q = t & 3;
    const int m = m0 + r;
    if (m >= a.m_rows) continue;  // uniform over the quad
    const u32x4 w = s_part[q * ROWS + r];
    RowStats st;
    st.m = __uint_as_float(w[0]);
    st.S = __uint_as_float(w[1]);
    st.T = __uint_as_float(w[2]);
    st.am = (int)w[3];
    st.merge_level<0>();
    st.merge_level<1>();
    if (q == 0)
      *reinterpret_cast<u32x4*>(a.partials + ((size_t)m * a.n_vtiles + vt) * kTileWords) =
          u32x4{__float_as_uint(st.m), __float_as_uint(st.S), __float_as_uint(st.T), (uint32_t)st.am};
  }
}

template <typename T, int MB>
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
  auto step_of = [&](int c) { return c + rot < n_steps ? c + rot : c + rot - n_steps; };
  const int v = min(vw + lr, a.vocab - 1);  // rows past V: a valid row, results not stored
  const char* wrow = reinterpret_cast<const char*>(a.w) + (size_t)v * row_bytes + lg * 16;
  const char* xbase = reinterpret_cast<const char*>(a.x);

  f32x4 acc[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) acc[mb] = f32x4{0.f, 0.f, 0.f, 0.f};

  // A ring of kStages K steps in registers: the W fragments and this thread's
  // share of the x tile of step c + kStages are requested together, right after
  // step c's products, so waiting for step c never waits for newer requests.
  // (Rows shorter than the ring: the slots past the last step are requested
  // with clamped steps and never consumed.)
  constexpr int kStages = MB == 3 ? 3 : 2;  // at most 256 VGPRs: two workgroups per CU
  constexpr int XPT = XStage<MB>::kPerThread;
  static_assert(XStage<MB>::kPieces % 256 == 0, "every thread stages whole pieces of x");
  struct Stage {
    u32x4 w[kLmPieces];
    u32x4 x[XPT];
  };
  auto issue = [&](Stage& st, int c) {
    const size_t off = (size_t)step_of(c) * kLmChunkBytes;
#pragma unroll
    for (int kp = 0; kp < kLmPieces; ++kp) st.w[kp] = ld16(wrow + off + kp * 64);
#pragma unroll
    for (int t = 0; t < XPT; ++t) {
      const int idx = threadIdx.x + 256 * t;
      const int r = idx / (kLmChunkBytes / 16), pc = idx % (kLmChunkBytes / 16);
      const int m = min(m0 + r, a.m_rows - 1);  // rows past M: a valid row, results not stored
      st.x[t] = ld16(xbase + (size_t)m * row_bytes + off + pc * 16);
    }
  };
  auto stage_x = [&](const Stage& st, unsigned char* buf) {
#pragma unroll
    for (int t = 0; t < XPT; ++t) {
      const int idx = threadIdx.x + 256 * t;
      const int r = idx / (kLmChunkBytes / 16), pc = idx % (kLmChunkBytes / 16);
      *reinterpret_cast<u32x4*>(buf + r * kLmXStride + pc * 16) = st.x[t];
    }
  };
  // x alternates between two LDS buffers: the barrier of step c+1 orders step
  // c's reads before the writes of step c+2
  auto step = [&](Stage& st, int c, bool refill) {
    unsigned char* buf = sx[c & 1];
    stage_x(st, buf);
    __syncthreads();
    mma_step<T, MB>(acc, st.w, buf, lr, lg);
    if (refill) issue(st, c + kStages);
    __builtin_amdgcn_sched_barrier(0);  // keep the requests here, ahead of the next step's wait
  };
  auto step_clamped = [&](Stage& st, int c) {
    unsigned char* buf = sx[c & 1];
    stage_x(st, buf);
    __syncthreads();
    mma_step<T, MB>(acc, st.w, buf, lr, lg);
    issue(st, min(c + kStages, n_steps - 1));
    __builtin_amdgcn_sched_barrier(0);
  };
  Stage ring[kStages];
#pragma unroll
  for (int j = 0; j < kStages; ++j) {
    issue(ring[j], min(j, n_steps - 1));
    __builtin_amdgcn_sched_barrier(0);
  }
  int c = 0;
  if constexpr (MB <= 2) {
    // Steady state: every step refills its slot with a real step, so the count
    // of requests behind every step is the same on every pass.  The last steps
    // (at most 2*kStages - 1, straight-line code) refill only while steps
    // remain: no request is left in flight at the end, where the epilogue's
    // barriers would wait for it (all workgroups of a small M run at once, so
    // that wait is not hidden behind other workgroups).
    for (; c + 2 * kStages <= n_steps; c += kStages) {
#pragma unroll
      for (int j = 0; j < kStages; ++j) step(ring[j], c + j, true);
    }
#pragma unroll
    for (int j = 0; j < 2 * kStages - 1; ++j)
      if (c + j < n_steps) step(ring[j % kStages], c + j, c + j + kStages < n_steps);
  } else {
    // (larger x tiles: past the last step the refills repeat the last step, unused,
    // which keeps the loop's register assignment stable)
    for (; c + kStages - 1 < n_steps; c += kStages) {
#pragma unroll
      for (int j = 0; j < kStages; ++j) step_clamped(ring[j], c + j);
    }
#pragma unroll
    for (int j = 0; j + 1 < kStages; ++j)
      if (c + j < n_steps) step_clamped(ring[j], c + j);
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
    tile_partials<MB>(acc, &sx[0][0], vw, vt, m0, a, lane, wave);
  }
}

// ---------------------------------------------------------------------------
// Persistent form of the same tile (large vocabularies): when the tiles
// outnumber the workgroups that fit on the GPU at once, each resident
// workgroup walks several tiles (ids blockIdx.x + k * gridDim.x) as one
// stream of K steps.  The register ring runs on across tile boundaries, so the
// next tile's first W steps are already in flight during a tile's epilogue,
// and there is one start-up latency per workgroup instead of one per tile.
// gridDim.x is a multiple of 8 * n_mtiles, so a workgroup keeps its M tile and
// the M tiles of one vocabulary tile still run together on one XCD; the ids
// past V all sit in the last group, so a workgroup's valid tiles are a prefix.
// Requires an even number of K steps per row (two ring slots per tile).
template <typename T, int MB>
__global__ __launch_bounds__(256, 2) void lmhead_persistent_kernel(LmArgs a) {
  constexpr int ES = Elem<T>::kBytes;
  __shared__ __align__(16) unsigned char sx[2][16 * MB * kLmXStride];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int n_mt = a.n_mtiles;
  const int n_vt = (a.vocab + kLmRows - 1) / kLmRows;
  const int n_ids = ((n_vt + 7) / 8) * 8 * n_mt;
  const int G = gridDim.x;
  auto vt_of = [&](int k) {
    const int id = (int)blockIdx.x + k * G;
    const int grp = id / (8 * n_mt), rem = id % (8 * n_mt);
    return grp * 8 + rem % 8;
  };
  int n_my = 0;
  while ((int)blockIdx.x + n_my * G < n_ids && vt_of(n_my) < n_vt) ++n_my;
  if (n_my == 0) return;
  const int mt = ((int)blockIdx.x % (8 * n_mt)) / 8;
  const int m0 = mt * 16 * MB;
  const size_t row_bytes = (size_t)a.hidden_size * ES;
  const int n_steps = (int)(row_bytes / kLmChunkBytes);
  const int total = n_my * n_steps;
  const char* xbase = reinterpret_cast<const char*>(a.x);
  const char* wbase = reinterpret_cast<const char*>(a.w);

  constexpr int XPT = XStage<MB>::kPerThread;
  static_assert(XStage<MB>::kPieces % 256 == 0, "every thread stages whole pieces of x");
  struct Stage {
    u32x4 w[kLmPieces];
    u32x4 x[XPT];
  };
  // global step g = k * n_steps + s: K step s of this workgroup's k-th tile
  // (each tile starts at its own rotated step, as in lmhead_kernel)
  auto issue = [&](Stage& st, int g) {
    const int k = g / n_steps, s = g - k * n_steps;
    const int vt = vt_of(k);
    const int rot = vt % n_steps;
    const size_t off = (size_t)(s + rot < n_steps ? s + rot : s + rot - n_steps) * kLmChunkBytes;
    const int v = min(vt * kLmRows + 16 * wave + lr, a.vocab - 1);  // rows past V: results not stored
    const char* wrow = wbase + (size_t)v * row_bytes + lg * 16;
#pragma unroll
    for (int kp = 0; kp < kLmPieces; ++kp) st.w[kp] = ld16(wrow + off + kp * 64);
#pragma unroll
    for (int t = 0; t < XPT; ++t) {
      const int idx = threadIdx.x + 256 * t;
      const int r = idx / (kLmChunkBytes / 16), pc = idx % (kLmChunkBytes / 16);
      const int m = min(m0 + r, a.m_rows - 1);  // rows past M: results not stored
      st.x[t] = ld16(xbase + (size_t)m * row_bytes + off + pc * 16);
    }
  };
  f32x4 acc[MB];
  auto step = [&](Stage& st, int g) {
    unsigned char* buf = sx[g & 1];
#pragma unroll
    for (int t = 0; t < XPT; ++t) {
      const int idx = threadIdx.x + 256 * t;
      const int r = idx / (kLmChunkBytes / 16), pc = idx % (kLmChunkBytes / 16);
      *reinterpret_cast<u32x4*>(buf + r * kLmXStride + pc * 16) = st.x[t];
    }
    __syncthreads();
    mma_step<T, MB>(acc, st.w, buf, lr, lg);
    issue(st, min(g + 2, total - 1));  // past the last step: the last step again, unused
    __builtin_amdgcn_sched_barrier(0);  // keep the requests here, ahead of the next step's wait
  };
  Stage ring[2];
  issue(ring[0], 0);
  __builtin_amdgcn_sched_barrier(0);
  issue(ring[1], min(1, total - 1));
  __builtin_amdgcn_sched_barrier(0);
  const bool vec_ok = (a.vocab & 3) == 0;
  for (int k = 0; k < n_my; ++k) {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int g0 = k * n_steps;
    for (int s = 0; s < n_steps; s += 2) {
      step(ring[0], g0 + s);
      step(ring[1], g0 + s + 1);
    }
    // epilogue of tile k (the next tile's first steps are already in flight)
    const int vt = vt_of(k);
    const int vw = vt * kLmRows + 16 * wave;
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
      tile_partials<MB>(acc, &sx[0][0], vw, vt, m0, a, lane, wave);
      __syncthreads();  // the statistics scratch is read before the next tile stages x
    }
  }
}

// ---------------------------------------------------------------------------
// GEMM variant (bf16), fed by DMA, in three tile shapes: MT = 256 token rows
// by VR = 128 vocabulary rows (129 or more rows in all), MT = 128 by VR = 128
// (65 to 128 rows), and MT = 64 by VR = 256 (at most 64 rows over a
// vocabulary of more than two 64-row tiles per CU, where each x row then
// serves four times as many W rows).  Every byte of W and x a workgroup needs
// crosses its CU once:
//   - K advances in 128-byte steps (64 elements); the W and x rows of a step go
//     straight from memory into an LDS stage by DMA (global_load_lds, 16 bytes
//     per lane, no registers), in a ring of S = 3 stages (48 or 40 KB): after the
//     barrier that publishes step c (every wave has finished step c-1 by then)
//     step c+2 is requested into c-1's stage, so two steps are in flight while
//     one is multiplied (the W and x rows of a step share a stage: giving W a
//     deeper register ring of its own measured slower);
//   - stage rows are 128 bytes with chunk c of row r stored at chunk position
//     c ^ ((r >> 1) & 7): a quarter-wave reading one chunk of 16 consecutive
//     rows touches all 64 banks once;
//   - eight waves (two per SIMD) in a WV x WT grid (VR/64 vocabulary waves;
//     token blocks past the last row are multiplied, not stored):
//     wave w owns vocabulary rows 64 (w % WV) .. +63 and token rows
//     MT/WT (w / WV) .. +MT/WT-1, and issues an eighth of every step's DMA
//     requests (at 256 x 128, four waves in a 2 x 2 grid, each with twice the
//     products and requests, measured ~6 % slower: the CU's feed from L2 grows
//     with the number of waves that issue);
//   - products on v_mfma_f32_32x32x16_bf16 with W as the A operand (32
//     vocabulary rows) and x as the B operand (32 token rows); each step's
//     fragments are requested ahead of its products;
//   - a lane's accumulator holds, for token row (lane & 31) of a block, the
//     vocabulary rows 8 g + 4 (lane >> 5) + e (g, e = 0..3) of a 32-row block;
//   - the logits leave through LDS as a [token row][VR] tile, so that each
//     token row's 4 VR bytes are stored contiguously, and each thread reduces
//     one token row of that tile over one 64-row statistics tile.
constexpr int kGmStep = 128;                    // bytes of a row per K step (64 elements)
constexpr int kGmWaves = 8;                     // waves per workgroup

template <int MT, int VR>
struct GmShape {
  static constexpr int WV = VR / 64;                                // vocabulary waves (64 rows each)
  static constexpr int WT = kGmWaves / WV;                          // token waves
  static constexpr int CPR = kGmStep / 16;                          // 16-byte chunks per stage row
  static constexpr int RPI = 64 / CPR;                              // stage rows per DMA request
  static constexpr int KS = kGmStep / 32;                           // 16-element slices per step
  static constexpr int kStage = (MT + VR) * kGmStep;                // bytes per stage
  static constexpr int S = 147456 / kStage;                         // stages (144 KB of LDS)
  static constexpr int kXInst = MT / RPI / kGmWaves;                // x DMA requests per wave per step
  static constexpr int kWInst = VR / RPI / kGmWaves;                // W DMA requests per wave per step
  static constexpr int kPerStep = kXInst + kWInst;
  static constexpr int NT = MT / WT / 32;                           // 32-row token blocks per wave
  static constexpr int kTileRowB = VR * 4 + 16;                     // LDS row stride of the logit tile
  static constexpr int kLds = S * kStage > MT * kTileRowB ? S * kStage : MT * kTileRowB;
  static constexpr int LPR = VR / 4;                                // lanes per token row of the store
  static constexpr int kStats = VR / kLmTileRows;                   // statistics tiles per token row
  static_assert(S >= 3 && (S - 1) * kPerStep <= 63, "stages and memory counter range");
  static_assert(VR % 64 == 0 && kGmWaves % WV == 0 && 64 % LPR == 0, "wave grid and store shape");
  static_assert(MT % (RPI * kGmWaves) == 0 && VR % (RPI * kGmWaves) == 0 && MT % (WT * 32) == 0,
                "every wave issues whole DMA requests and owns whole 32-row token blocks");
  // chunk position of chunk c of stage row r
  static __device__ __forceinline__ int swz(int c, int r) { return c ^ ((r >> 1) & 7); }
};

// One 1 KB DMA request (8 rows of 128 bytes): lane l fills chunk position l % 8
// of row 8 q + l / 8 with the chunk that belongs there.
__device__ __forceinline__ void gm_dma(uint32_t lds_dst, uint64_t base, uint32_t off) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %2, %3\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(lds_dst), "v"(off), "s"(base)
      : "memory");
}

__device__ __forceinline__ uint64_t uniform_u64(uint64_t v) {
  return ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(v >> 32)) << 32) |
         (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)v);
}

template <int MT, int VR>
__global__ __launch_bounds__(64 * kGmWaves) void lmhead_gemm_kernel(LmArgs a) {
  using G = GmShape<MT, VR>;
  typedef float f32x16 __attribute__((ext_vector_type(16)));
  __shared__ __align__(1024) unsigned char sm[G::kLds];
  const uint32_t lds0 = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) unsigned char*)sm;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r32 = lane & 31, hi = lane >> 5;
  const int n_mt = a.n_mtiles;
  const int id = blockIdx.x;
  const int grp = id / (8 * n_mt), rem = id % (8 * n_mt);
  const int vt = grp * 8 + rem % 8, mt = rem / 8;  // the M tiles of a vocabulary tile share an XCD
  if (vt * VR >= a.vocab) return;
  const int v0 = vt * VR;
  const int m0 = mt * MT;
  const size_t row_bytes = (size_t)a.hidden_size * 2;
  const int n_steps = (int)(row_bytes / kGmStep);  // >= 4 (hidden*2 is a multiple of 512; checked)
  // K start: four phases, by vocabulary tile / 8 mod 4, so that the 32
  // workgroups on one XCD (tiles congruent mod 8) stream x from four points
  // (all from one point, or one each, measured slower)
  const int rot = ((vt >> 3) & 3) * (n_steps / 4);

  // this lane's DMA offsets (rows past M or V read a valid row; results not stored)
  uint32_t xo[G::kXInst], wo[G::kWInst];
#pragma unroll
  for (int j = 0; j < G::kXInst; ++j) {
    const int r = G::RPI * (wave * G::kXInst + j) + lane / G::CPR, pos = lane % G::CPR;
    const int m = min(m0 + r, a.m_rows - 1);
    xo[j] = (uint32_t)((size_t)(m - m0) * row_bytes + G::swz(pos, r) * 16);
  }
#pragma unroll
  for (int j = 0; j < G::kWInst; ++j) {
    const int r = G::RPI * (wave * G::kWInst + j) + lane / G::CPR, pos = lane % G::CPR;
    const int v = min(v0 + r, a.vocab - 1);
    wo[j] = (uint32_t)((size_t)(v - v0) * row_bytes + G::swz(pos, r) * 16);
  }
  const uint64_t xbase = reinterpret_cast<uint64_t>(a.x) + (uint64_t)m0 * row_bytes;
  const uint64_t wbase = reinterpret_cast<uint64_t>(a.w) + (uint64_t)v0 * row_bytes;
  auto issue = [&](int c) {  // requests of step c into stage c % S
    const int kc = c + rot < n_steps ? c + rot : c + rot - n_steps;
    const uint64_t ko = (uint64_t)kc * kGmStep;
    const uint32_t st = lds0 + (uint32_t)((c % G::S) * G::kStage);
    const uint64_t xb = uniform_u64(xbase + ko), wb = uniform_u64(wbase + ko);
#pragma unroll
    for (int j = 0; j < G::kXInst; ++j)
      gm_dma(__builtin_amdgcn_readfirstlane(st + (uint32_t)((wave * G::kXInst + j) * 1024)), xb, xo[j]);
#pragma unroll
    for (int j = 0; j < G::kWInst; ++j)
      gm_dma(__builtin_amdgcn_readfirstlane(st + (uint32_t)(MT * kGmStep + (wave * G::kWInst + j) * 1024)), wb,
             wo[j]);
  };

  const int wv = wave % G::WV, wt = wave / G::WV;
  // LDS byte offsets of this lane's fragments within a 32-row block, per 16-element slice
  uint32_t kof[G::KS];
#pragma unroll
  for (int ks = 0; ks < G::KS; ++ks) kof[ks] = (uint32_t)(r32 * kGmStep + G::swz(2 * ks + hi, r32) * 16);
  const int a_row0 = MT + 64 * wv;     // stage row of the wave's first W row
  const int b_row0 = wt * (MT / G::WT);  // stage row of the wave's first x row

  f32x16 acc[2][G::NT];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int n = 0; n < G::NT; ++n) acc[i][n] = f32x16{};

#pragma unroll
  for (int j = 0; j < G::S - 1; ++j)
    if (j < n_steps) issue(j);
  for (int c = 0; c < n_steps; ++c) {
    // step c's own requests have landed once at most the newer steps' are pending
    if (c + G::S - 2 < n_steps)
      asm volatile("s_waitcnt vmcnt(%0)\n\ts_waitcnt lgkmcnt(0)\n\ts_barrier" ::"n"((G::S - 2) * G::kPerStep)
                   : "memory");
    else
      asm volatile("s_waitcnt vmcnt(0)\n\ts_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    if (c + G::S - 1 < n_steps) issue(c + G::S - 1);  // into the stage step c-1 used
    const unsigned char* st = sm + (c % G::S) * G::kStage;
    // (token blocks past the last row are multiplied too: clamped rows, not stored)
    u32x4 af[G::KS][2], bfr[G::KS][G::NT];
#pragma unroll
    for (int ks = 0; ks < G::KS; ++ks) {
#pragma unroll
      for (int i = 0; i < 2; ++i)
        af[ks][i] = *reinterpret_cast<const u32x4*>(st + (a_row0 + 32 * i) * kGmStep + kof[ks]);
#pragma unroll
      for (int n = 0; n < G::NT; ++n)
        bfr[ks][n] = *reinterpret_cast<const u32x4*>(st + (b_row0 + 32 * n) * kGmStep + kof[ks]);
    }
#pragma unroll
    for (int ks = 0; ks < G::KS; ++ks)
#pragma unroll
      for (int n = 0; n < G::NT; ++n)
#pragma unroll
        for (int i = 0; i < 2; ++i)
          acc[i][n] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, af[ks][i]),
                                                              __builtin_bit_cast(bf16x8, bfr[ks][n]), acc[i][n], 0, 0, 0);
    // schedule: the reads of slices 0 and 1, then each slice's products behind
    // the reads of the slice after next
    constexpr int kRd = 2 + G::NT, kMm = 2 * G::NT;
    __builtin_amdgcn_sched_group_barrier(0x100, 2 * kRd, 0);
#pragma unroll
    for (int ks = 0; ks + 2 < G::KS; ++ks) {
      __builtin_amdgcn_sched_group_barrier(0x008, kMm, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, kRd, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x008, 2 * kMm, 0);
  }

  // logits through LDS: the stages are free once every wave has finished the last step
  __syncthreads();
  unsigned char* tile = sm;  // [MT][kTileRowB] bytes
#pragma unroll
  for (int n = 0; n < G::NT; ++n)
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int row = b_row0 + 32 * n + r32, col = 64 * wv + 32 * i + 8 * g + 4 * hi;
        *reinterpret_cast<f32x4*>(tile + row * G::kTileRowB + col * 4) =
            f32x4{acc[i][n][4 * g], acc[i][n][4 * g + 1], acc[i][n][4 * g + 2], acc[i][n][4 * g + 3]};
      }
  __syncthreads();
  const int rows = min(MT, a.m_rows - m0);
  {
    const bool vec_ok = (a.vocab & 3) == 0;
    constexpr int kRowsPerWave = 64 / G::LPR;  // token rows a wave stores per pass
    const int col = 4 * (lane % G::LPR);        // this lane's 4 vocabulary rows of a token row
    const int vv = v0 + col;
    for (int row = kRowsPerWave * wave + lane / G::LPR; row < rows; row += kRowsPerWave * kGmWaves) {
      const f32x4 q = *reinterpret_cast<const f32x4*>(tile + row * G::kTileRowB + col * 4);
      float* dst = a.logits + (size_t)(m0 + row) * a.vocab + vv;
      if (vec_ok && vv + 3 < a.vocab) {
        *reinterpret_cast<f32x4*>(dst) = q;
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (vv + e < a.vocab) dst[e] = q[e];
      }
    }
  }
  if (!a.partials) return;

  // statistics: one (token row, 64-row statistics tile) pair per thread and pass
  for (int u = threadIdx.x; u < MT * G::kStats; u += 64 * kGmWaves) {
    {
      const int row = u % MT, h = u / MT;
      const int vh = v0 + kLmTileRows * h;
      if (row >= rows || vh >= a.vocab) continue;  // (no statistics tile past V)
      const unsigned char* zr = tile + row * G::kTileRowB + h * kLmTileRows * 4;
      float z[kLmTileRows];
#pragma unroll
      for (int q = 0; q < kLmTileRows / 4; ++q) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(zr + 16 * q);
        z[4 * q] = v[0];
        z[4 * q + 1] = v[1];
        z[4 * q + 2] = v[2];
        z[4 * q + 3] = v[3];
      }
      const int nv = a.vocab - vh;  // entries at or past V are not logits
      float mx = kNegInf;
#pragma unroll
      for (int i = 0; i < kLmTileRows; ++i) mx = i < nv ? fmaxf(mx, z[i]) : mx;
      float S = 0.f, T = 0.f;
      int am = 0x7FFFFFFF;
#pragma unroll
      for (int i = kLmTileRows - 1; i >= 0; --i) {
        const bool ok = i < nv;
        const float d = z[i] - mx;
        const float e = ok ? __expf(d) : 0.f;
        S += e;
        T += ok ? e * d : 0.f;
        am = (ok && z[i] == mx) ? vh + i : am;
      }
      *reinterpret_cast<u32x4*>(a.partials + ((size_t)(m0 + row) * a.n_vtiles + vh / kLmTileRows) * kTileWords) =
          u32x4{__float_as_uint(mx), __float_as_uint(S), __float_as_uint(T), (uint32_t)am};
    }
  }
}

// Workgroups of a kernel that fit on the device at once (host occupancy
// query, cached per kernel; 0 if the query fails).
template <typename F>
static int resident_wgs(F kernel) {
  static std::atomic<int> cached{-1};
  int v = cached.load(std::memory_order_relaxed);
  if (v >= 0) return v;
  int per_cu = 0, dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void*>(kernel), 256, 0) !=
          hipSuccess)
    v = 0;
  else
    v = per_cu * cus;
  cached.store(v, std::memory_order_relaxed);
  return v;
}

template <typename T, int MB>
static hipError_t launch_plain(dim3 grid, const LmArgs& a, hipStream_t s, hipEvent_t ev_stop) {
  const dim3 blk(256);
  const int n_steps = (int)((size_t)a.hidden_size * Elem<T>::kBytes / kLmChunkBytes);
  const int unit = 8 * a.n_mtiles;  // the persistent grid keeps whole groups of 8 vocabulary tiles
  const int slots = resident_wgs(lmhead_persistent_kernel<T, MB>) / unit * unit;
  if (n_steps % 2 == 0 && slots >= unit && (int)grid.x > slots)
    return launch_k(lmhead_persistent_kernel<T, MB>, dim3(slots), blk, 0, s, nullptr, ev_stop, a);
  return launch_k(lmhead_kernel<T, MB>, grid, blk, 0, s, nullptr, ev_stop, a);
}

template <typename T>
static hipError_t launch_mb(int mb, dim3 grid, const LmArgs& a, hipStream_t s, hipEvent_t ev_stop) {
  switch (mb) {
    case 1: return launch_plain<T, 1>(grid, a, s, ev_stop);
    case 2: return launch_plain<T, 2>(grid, a, s, ev_stop);
    case 3: return launch_plain<T, 3>(grid, a, s, ev_stop);
    case 4: return launch_plain<T, 4>(grid, a, s, ev_stop);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_lmhead(int dtype, int mb, bool wide, const LmArgs& a, hipStream_t s, hipEvent_t ev_stop) {
  const int n_vt = (a.vocab + kLmRows - 1) / kLmRows;
  const int n_grp = (n_vt + 7) / 8;
  dim3 grid(n_grp * 8 * a.n_mtiles);
  if (mb == 8) {  // GEMM variant: 128 token rows per tile, 128-row vocabulary tiles (bf16)
    if (dtype != 1 || a.hidden_size % 256 != 0) return hipErrorInvalidValue;
    const int n_vt2 = (a.vocab + 127) / 128;
    dim3 tgrid(((n_vt2 + 7) / 8) * 8 * a.n_mtiles);
    return launch_k(lmhead_gemm_kernel<128, 128>, tgrid, dim3(64 * kGmWaves), 0, s, nullptr, ev_stop, a);
  }
  if (mb == 16) {  // GEMM variant: 256 token rows per tile, 128-row vocabulary tiles (bf16)
    if (dtype != 1 || a.hidden_size % 256 != 0) return hipErrorInvalidValue;
    const int n_vt2 = (a.vocab + 127) / 128;
    dim3 tgrid(((n_vt2 + 7) / 8) * 8 * a.n_mtiles);
    return launch_k(lmhead_gemm_kernel<256, 128>, tgrid, dim3(64 * kGmWaves), 0, s, nullptr, ev_stop, a);
  }
  if (wide) {  // GEMM variant: up to 64 token rows, 256-row vocabulary tiles (bf16)
    if (dtype != 1 || mb > 4 || a.hidden_size % 256 != 0) return hipErrorInvalidValue;
    const int n_vt2 = (a.vocab + 255) / 256;
    dim3 tgrid(((n_vt2 + 7) / 8) * 8 * a.n_mtiles);
    return launch_k(lmhead_gemm_kernel<64, 256>, tgrid, dim3(64 * kGmWaves), 0, s, nullptr, ev_stop, a);
  }
  return dtype == 1 ? launch_mb<bf16_t>(mb, grid, a, s, ev_stop) : launch_mb<float>(mb, grid, a, s, ev_stop);
}

}  // namespace respec
