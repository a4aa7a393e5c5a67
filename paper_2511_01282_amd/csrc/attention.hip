// Tree-masked grouped-query attention of draft-tree nodes against the KV cache,
// fused with the split merge and the residual x = round(h + O).
//
// This is the target's parallel verification forward over a draft tree
// (ReSpec, Section 3.5 / Algorithm 1), reduced to one attention layer: node i
// attends to every prefix row of its sequence and to the tree rows of its
// ancestors and itself.
//
// Work decomposition (one workgroup per (sequence b, KV head g, row block, KV
// split)):
//   - query rows of a KV head are (node, head-in-group) pairs, r = node*G + hh;
//     a wave owns 16*NB of them, a workgroup wr*(16*NB); its wk wave columns
//     share the split's KV rows in 32-row steps;
//   - S^T = K Q^T on the matrix cores (K fragments straight from HBM, Q held in
//     registers for the whole loop), online softmax in log2 units;
//   - V is transposed through a per-wave LDS tile so that O^T = V^T P^T runs on
//     the matrix cores; bf16 P is split into hi + lo bf16 parts so that the
//     probabilities keep ~16 significant bits (bf16 P alone perturbs x enough
//     to move logits by ~5e-4);
//   - waves of a row group are merged in LDS; each workgroup writes an
//     unnormalised partial (O, max, sum) with device-coherent stores; the last
//     workgroup of a (b, g, row block) to finish (device-scope ticket) merges
//     all splits, writes O and x, and resets the ticket to zero for the next
//     step.
#include "common.hpp"
#include "kernels.hpp"

namespace respec {

template <typename T, int D>
struct AttnTile {
  static constexpr int ES = Elem<T>::kBytes;
  static constexpr int KCH = D * ES / 64;  // 64-byte K-chunks per head row
  static constexpr int CPR = D * ES / 16;  // 16-byte pieces per KV row
  static constexpr int VPL = CPR / 8;      // (piece, 4-row quad) pairs per lane per tile
  u32x4 k[2][KCH];                         // K rows t0 + 16*kb + lr, this lane's pieces
  u32x4 v[VPL][4];                         // V piece c of rows t0 + 4*qd + r
};

// Issue the global loads of one 32-row KV tile.  Rows at or beyond kv_hi are
// clamped to kv_hi - 1 (a valid row of this split): their scores are masked
// and their values are multiplied by zero probabilities.
template <typename T, int D>
__device__ __forceinline__ void load_tile(AttnTile<T, D>& t, const char* kbase, const char* vbase, int t0, int kv_hi,
                                          int lane) {
  using A = AttnTile<T, D>;
  const int lr = lane & 15, lg = lane >> 4;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    const int p = min(t0 + 16 * kb + lr, kv_hi - 1);
    const char* src = kbase + (size_t)p * D * A::ES;
#pragma unroll
    for (int kc = 0; kc < A::KCH; ++kc) t.k[kb][kc] = ld16(src + kc * 64 + lg * 16);
  }
#pragma unroll
  for (int q = 0; q < A::VPL; ++q) {
    const int pair = lane + 64 * q;
    const int c = pair % A::CPR, qd = pair / A::CPR;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int p = min(t0 + 4 * qd + r, kv_hi - 1);
      t.v[q][r] = ld16(vbase + (size_t)p * D * A::ES + c * 16);
    }
  }
}

// Online-softmax attention of this wave's query rows over one loaded tile.
// Scores stay unscaled until the exponent: p = 2^(s * scale_log2 - m).
template <typename T, int D, int NB>
__device__ __forceinline__ void process_tile(const AttnTile<T, D>& t, int t0, int kv_hi, int L, T* vt,
                                             const u32x4 (&qf)[NB][D * Elem<T>::kBytes / 64], const int (&qnode)[NB],
                                             const uint32_t* s_anc, float scale_log2, float (&m_run)[NB],
                                             float (&l_run)[NB], f32x4 (&o)[D / 16][NB], int lane) {
  using A = AttnTile<T, D>;
  constexpr int ES = A::ES;
  constexpr int E16 = 16 / ES;
  constexpr int DB = D / 16;
  constexpr int VTS = kKvTile + kVtPad;
  const int lr = lane & 15, lg = lane >> 4;

  // write V^T: vt[d][kv] (4 consecutive kv per 8-byte / 16-byte store)
#pragma unroll
  for (int q = 0; q < A::VPL; ++q) {
    const int pair = lane + 64 * q;
    const int c = pair % A::CPR, qd = pair / A::CPR;
    if constexpr (ES == 2) {
#pragma unroll
      for (int w = 0; w < 4; ++w) {  // word w holds d = c*8 + 2w (low half) and 2w+1 (high half)
        const uint32_t r0 = t.v[q][0][w], r1 = t.v[q][1][w], r2 = t.v[q][2][w], r3 = t.v[q][3][w];
        const u32x2 even = {__builtin_amdgcn_perm(r1, r0, 0x05040100u), __builtin_amdgcn_perm(r3, r2, 0x05040100u)};
        const u32x2 odd = {__builtin_amdgcn_perm(r1, r0, 0x07060302u), __builtin_amdgcn_perm(r3, r2, 0x07060302u)};
        *reinterpret_cast<u32x2*>(vt + (c * E16 + 2 * w) * VTS + 4 * qd) = even;
        *reinterpret_cast<u32x2*>(vt + (c * E16 + 2 * w + 1) * VTS + 4 * qd) = odd;
      }
    } else {
#pragma unroll
      for (int e = 0; e < E16; ++e)
        *reinterpret_cast<u32x4*>(vt + (c * E16 + e) * VTS + 4 * qd) =
            u32x4{t.v[q][0][e], t.v[q][1][e], t.v[q][2][e], t.v[q][3][e]};
    }
  }
  wave_lds_sync();

  // S^T = K Q^T: lane holds S[query 16*nb + lr][kv t0 + 16*kb + 4*lg + i] (unscaled)
  f32x4 s[2][NB];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kc = 0; kc < A::KCH; ++kc) acc = mma_k64(T{}, t.k[kb][kc], qf[nb][kc], acc);
      s[kb][nb] = acc;
    }
  }
  // tree mask and range mask, only for tiles that reach the tree rows or the split end
  if (t0 + kKvTile > kv_hi || t0 + kKvTile > L) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int p = t0 + 16 * kb + 4 * lg + i;
        const int ai = p - L;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          bool vis = p < kv_hi;
          if (vis && ai >= 0) vis = qnode[nb] >= 0 && ((s_anc[qnode[nb] * 4 + (ai >> 5)] >> (ai & 31)) & 1u);
          s[kb][nb][i] = vis ? s[kb][nb][i] : kNegInf;
        }
      }
    }
  }
  // online softmax (row max shared by the 4 lane groups of a row)
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    float tm = kNegInf;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) tm = fmaxf(tm, fmaxf(fmaxf(s[kb][nb][0], s[kb][nb][1]), fmaxf(s[kb][nb][2], s[kb][nb][3])));
    tm = fmaxf(tm, __shfl_xor(tm, 16, 64));
    tm = fmaxf(tm, __shfl_xor(tm, 32, 64));
    const float mn = fmaxf(m_run[nb], tm * scale_log2);
    const bool none = mn == kNegInf;
    const float alpha = none ? 1.f : __builtin_amdgcn_exp2f(m_run[nb] - mn);
    const float mb = none ? 0.f : mn;
    float ps = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float pv = __builtin_amdgcn_exp2f(__builtin_fmaf(s[kb][nb][i], scale_log2, -mb));
        s[kb][nb][i] = pv;
        ps += pv;
      }
    l_run[nb] = l_run[nb] * alpha + ps;
    m_run[nb] = mn;
    if (__any(alpha != 1.f)) {
#pragma unroll
      for (int db = 0; db < DB; ++db) o[db][nb] *= alpha;
    }
  }

  // O^T += V^T P^T: k order per lane = kv {4lg+i (kb 0), 16+4lg+i (kb 1)}
  if constexpr (ES == 2) {
    typedef float f32x2 __attribute__((ext_vector_type(2)));
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    u32x4 phi[NB], plo[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float p0 = s[j >> 1][nb][2 * (j & 1)], p1 = s[j >> 1][nb][2 * (j & 1) + 1];
        const uint32_t h = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{p0, p1}, bf16x2));
        const float r0 = p0 - __uint_as_float(h << 16), r1 = p1 - __uint_as_float(h & 0xFFFF0000u);
        phi[nb][j] = h;
        plo[nb][j] = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{r0, r1}, bf16x2));
      }
    }
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const T* row = vt + (16 * db + lr) * VTS;
      const u32x2 v0 = *reinterpret_cast<const u32x2*>(row + 4 * lg);
      const u32x2 v1 = *reinterpret_cast<const u32x2*>(row + 16 + 4 * lg);
      const u32x4 af = {v0.x, v0.y, v1.x, v1.y};
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        o[db][nb] = mma_k64(T{}, af, phi[nb], o[db][nb]);
        o[db][nb] = mma_k64(T{}, af, plo[nb], o[db][nb]);
      }
    }
  } else {
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const T* row = vt + (16 * db + lr) * VTS;
      const f32x4 v0 = *reinterpret_cast<const f32x4*>(row + 4 * lg);
      const f32x4 v1 = *reinterpret_cast<const f32x4*>(row + 16 + 4 * lg);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          o[db][nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(v0[i], s[0][nb][i], o[db][nb], 0, 0, 0);
#pragma unroll
        for (int i = 0; i < 4; ++i)
          o[db][nb] = __builtin_amdgcn_mfma_f32_16x16x4f32(v1[i], s[1][nb][i], o[db][nb], 0, 0, 0);
      }
    }
  }
  wave_lds_sync();  // this tile's V^T reads precede the next tile's writes
}

// ---------------------------------------------------------------------------
// bf16 path: V tiles go HBM -> LDS by DMA (global_load_lds, 16 bytes per lane,
// no registers) and are read back transposed with ds_read_b64_tr_b16.
//
// LDS tile layout: 32 rows x D bf16, row-major; 16-byte chunk c of row r is
// stored at chunk position c ^ vswz(r) so that the transposing reads of a
// half-wave (8 rows x 2 chunks each) hit 64 distinct banks.
// Transposing read: within a 16-lane group, lane i receives element i%4 of the
// 8-byte pieces addressed by lanes i/4 + 4e (e = 0..3).  Lane j of group lg
// addresses row 16*kb + 4*lg + j/4, columns 16*db + 4*(j%4) .. +3, so lane lr
// receives V[16*kb + 4*lg + e][16*db + lr], e = 0..3: the A operand of
// O^T = V^T P^T in the kv order the P fragments use.
template <int D>
__device__ __forceinline__ int vswz(int r) {
  return D == 128 ? ((2 * r) & 14) : (r & 6);
}

template <int D>
struct KTile {
  static constexpr int KCH = D * 2 / 64;
  u32x4 k[2][KCH];
};

template <int D>
__device__ __forceinline__ void load_k_bf16(KTile<D>& t, const char* kbase, int t0, int kv_hi, int lane) {
  const int lr = lane & 15, lg = lane >> 4;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    const int p = min(t0 + 16 * kb + lr, kv_hi - 1);
    const char* src = kbase + (size_t)p * D * 2;
#pragma unroll
    for (int kc = 0; kc < KTile<D>::KCH; ++kc) t.k[kb][kc] = ld16(src + kc * 64 + lg * 16);
  }
}

// DMA one 32-row V tile into the wave's LDS tile (rows >= kv_hi clamped).
template <int D>
__device__ __forceinline__ void dma_v_bf16(unsigned char* vtile, const char* vbase, int t0, int kv_hi, int lane) {
  constexpr int CPR = D * 2 / 16;      // 16-byte chunks per row
  constexpr int RPI = 64 / CPR;        // rows per DMA instruction
#pragma unroll
  for (int q = 0; q < kKvTile / RPI; ++q) {
    const int r = q * RPI + lane / CPR, slot = lane % CPR;
    const int p = min(t0 + r, kv_hi - 1);
    const char* src = vbase + (size_t)p * D * 2 + (size_t)(slot ^ vswz<D>(r)) * 16;
    __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)src,
                                     (__attribute__((address_space(3))) void*)(vtile + q * 1024), 16, 0, 0);
  }
}

template <int D, int NB>
__device__ __forceinline__ void process_tile_bf16(const KTile<D>& t, const unsigned char* vtile, int t0, int kv_hi,
                                                  int L, const u32x4 (&qf)[NB][D * 2 / 64], const int (&qnode)[NB],
                                                  const uint32_t* s_anc, float scale_log2, float (&m_run)[NB],
                                                  float (&l_run)[NB], f32x4 (&o)[D / 16][NB], int lane) {
  constexpr int KCH = D * 2 / 64;
  constexpr int DB = D / 16;
  const int lr = lane & 15, lg = lane >> 4;
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

  // S^T = K Q^T (unscaled)
  f32x4 s[2][NB];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kc = 0; kc < KCH; ++kc) acc = mma_k64(bf16_t{}, t.k[kb][kc], qf[nb][kc], acc);
      s[kb][nb] = acc;
    }
  }
  if (t0 + kKvTile > kv_hi || t0 + kKvTile > L) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int p = t0 + 16 * kb + 4 * lg + i;
        const int ai = p - L;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          bool vis = p < kv_hi;
          if (vis && ai >= 0) vis = qnode[nb] >= 0 && ((s_anc[qnode[nb] * 4 + (ai >> 5)] >> (ai & 31)) & 1u);
          s[kb][nb][i] = vis ? s[kb][nb][i] : kNegInf;
        }
      }
    }
  }
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    float tm = kNegInf;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
      tm = fmaxf(tm, fmaxf(fmaxf(s[kb][nb][0], s[kb][nb][1]), fmaxf(s[kb][nb][2], s[kb][nb][3])));
    tm = fmaxf(tm, __shfl_xor(tm, 16, 64));
    tm = fmaxf(tm, __shfl_xor(tm, 32, 64));
    const float mn = fmaxf(m_run[nb], tm * scale_log2);
    const bool none = mn == kNegInf;
    const float alpha = none ? 1.f : __builtin_amdgcn_exp2f(m_run[nb] - mn);
    const float mb = none ? 0.f : mn;
    float ps = 0.f;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float pv = __builtin_amdgcn_exp2f(__builtin_fmaf(s[kb][nb][i], scale_log2, -mb));
        s[kb][nb][i] = pv;
        ps += pv;
      }
    l_run[nb] = l_run[nb] * alpha + ps;
    m_run[nb] = mn;
    if (__any(alpha != 1.f)) {
#pragma unroll
      for (int db = 0; db < DB; ++db) o[db][nb] *= alpha;
    }
  }
  // P^T fragments, hi + lo bf16 parts
  u32x4 phi[NB], plo[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float p0 = s[j >> 1][nb][2 * (j & 1)], p1 = s[j >> 1][nb][2 * (j & 1) + 1];
      const uint32_t h = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{p0, p1}, bf16x2));
      const float r0 = p0 - __uint_as_float(h << 16), r1 = p1 - __uint_as_float(h & 0xFFFF0000u);
      phi[nb][j] = h;
      plo[nb][j] = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{r0, r1}, bf16x2));
    }
  }
  // V^T fragments by transposing LDS reads
  const int j = lr;
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    u32x2 half[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const int r = 16 * kb + 4 * lg + j / 4;
      const int col = 16 * db + 4 * (j % 4);
      const int chunk = (col >> 3) ^ vswz<D>(r);
      const unsigned char* addr = vtile + r * (D * 2) + chunk * 16 + (col & 7) * 2;
      const bf16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(addr));
      half[kb] = __builtin_bit_cast(u32x2, v);
    }
    const u32x4 af = {half[0].x, half[0].y, half[1].x, half[1].y};
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      o[db][nb] = mma_k64(bf16_t{}, af, phi[nb], o[db][nb]);
      o[db][nb] = mma_k64(bf16_t{}, af, plo[nb], o[db][nb]);
    }
  }
}

template <typename T, int D, int NB>
__global__ __launch_bounds__(256) void tree_attn_kernel(AttnArgs a) {
  constexpr int ES = Elem<T>::kBytes;
  constexpr int KCH = D * ES / 64;     // 64-byte K-chunks per head row
  constexpr int DB = D / 16;           // 16-wide output blocks along D
  constexpr int VTS = kKvTile + kVtPad;  // elements per transposed-V row
  constexpr int RB = 16 * NB;          // query rows per wave

  extern __shared__ __align__(16) unsigned char smem[];
  uint32_t* s_anc = reinterpret_cast<uint32_t*>(smem);                 // [kMaxNodes][4]
  int* s_par = reinterpret_cast<int*>(smem + kMaxNodes * 16);          // [kMaxNodes]
  int* s_ticket = reinterpret_cast<int*>(smem + kMaxNodes * 20);       // [1]
  unsigned char* s_work = smem + kMaxNodes * 20 + 64;

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int nwaves = blockDim.x >> 6;
  const int wr = wave % a.wr, wk = wave / a.wr;
  const int b = blockIdx.z;
  const int g = blockIdx.y / a.n_rowblk, rb = blockIdx.y % a.n_rowblk;
  const int split = blockIdx.x;

  // Sequence bounds; invalid device data degrades to an empty sequence.
  const int node0 = a.node_off[b], node1 = a.node_off[b + 1];
  int n_nodes = node1 - node0;
  if (node0 < 0 || node1 > a.total_nodes || n_nodes < 1 || n_nodes > a.max_nodes) n_nodes = 0;
  int L = a.kv_len[b];
  L = max(0, min(L, a.kv_cap - n_nodes));
  const int R = n_nodes * a.group;
  const int row_wg = rb * a.rows_per_wg;
  if (row_wg >= R) return;  // uniform over every split of this row block

  const size_t head_row0 = ((size_t)b * a.n_kv_heads + g) * (size_t)a.kv_cap;
  const char* kbase = reinterpret_cast<const char*>(a.k_cache) + head_row0 * D * ES;
  const char* vbase = reinterpret_cast<const char*>(a.v_cache) + head_row0 * D * ES;
  const int t_rows = L + n_nodes;
  const int kv_lo = split * a.chunk;
  const int kv_hi = min(kv_lo + a.chunk, t_rows);
  const int t_first = kv_lo + wk * kKvTile, t_step = kKvTile * a.wk;

  // Query fragments (lane row r = row_wave + 16*nb + lr) and the first tile, issued first.
  const int row_wave = row_wg + wr * RB;
  u32x4 qf[NB][KCH];
  int qnode[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int r = row_wave + 16 * nb + lr;
    qnode[nb] = -1;
    if (r < R) {
      const int node = r / a.group;
      const int h = g * a.group + (r - node * a.group);
      qnode[nb] = node;
      const char* src = reinterpret_cast<const char*>(a.hidden) +
                        ((size_t)(node0 + node) * a.hidden_size + (size_t)h * D) * ES;
#pragma unroll
      for (int kc = 0; kc < KCH; ++kc) qf[nb][kc] = ld16(src + kc * 64 + lg * 16);
    } else {
#pragma unroll
      for (int kc = 0; kc < KCH; ++kc) qf[nb][kc] = u32x4{0, 0, 0, 0};
    }
  }
  [[maybe_unused]] AttnTile<T, D> ta;
  [[maybe_unused]] AttnTile<T, D> tb;
  [[maybe_unused]] KTile<D> ka;
  [[maybe_unused]] KTile<D> kb2;
  unsigned char* vtiles = s_work + (size_t)wave * 2 * kKvTile * D * ES;  // bf16: two V tiles per wave
  if constexpr (ES == 2) {
    if (t_first < kv_hi) {
      load_k_bf16<D>(ka, kbase, t_first, kv_hi, lane);
      dma_v_bf16<D>(vtiles, vbase, t_first, kv_hi, lane);
    }
  } else {
    if (t_first < kv_hi) load_tile<T, D>(ta, kbase, vbase, t_first, kv_hi, lane);
  }

  // Ancestor-or-self bitsets of the sequence's nodes, from the parent array in LDS.
  for (int t = threadIdx.x; t < n_nodes; t += blockDim.x) s_par[t] = a.parent[node0 + t];
  __syncthreads();
  for (int t = threadIdx.x; t < n_nodes; t += blockDim.x) {
    uint32_t w0 = 0, w1 = 0, w2 = 0, w3 = 0;
    int x = t;
    for (int step = 0; step < kMaxNodes; ++step) {
      const uint32_t bit = 1u << (x & 31);
      const int word = x >> 5;
      w0 |= word == 0 ? bit : 0u;
      w1 |= word == 1 ? bit : 0u;
      w2 |= word == 2 ? bit : 0u;
      w3 |= word == 3 ? bit : 0u;
      if (x == 0) break;
      const int p = s_par[x];
      if (p < 0 || p >= x) break;
      x = p;
    }
    s_anc[t * 4 + 0] = w0;
    s_anc[t * 4 + 1] = w1;
    s_anc[t * 4 + 2] = w2;
    s_anc[t * 4 + 3] = w3;
  }
  __syncthreads();

  float m_run[NB], l_run[NB];
  f32x4 o[DB][NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    m_run[nb] = kNegInf;
    l_run[nb] = 0.f;
#pragma unroll
    for (int db = 0; db < DB; ++db) o[db][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  if constexpr (ES == 2) {
    // Two tiles in flight: wait for tile k (K in registers, V in LDS), issue tile k+1, process k.
    constexpr int VT = kKvTile * D * 2;
    for (int t0 = t_first; t0 < kv_hi; t0 += 2 * t_step) {
      const int t1 = t0 + t_step;
      __builtin_amdgcn_s_waitcnt(0);
      wave_lds_sync();
      if (t1 < kv_hi) {
        load_k_bf16<D>(kb2, kbase, t1, kv_hi, lane);
        dma_v_bf16<D>(vtiles + VT, vbase, t1, kv_hi, lane);
      }
      process_tile_bf16<D, NB>(ka, vtiles, t0, kv_hi, L, qf, qnode, s_anc, a.scale_log2, m_run, l_run, o, lane);
      if (t1 >= kv_hi) break;
      const int t2 = t1 + t_step;
      __builtin_amdgcn_s_waitcnt(0);
      wave_lds_sync();
      if (t2 < kv_hi) {
        load_k_bf16<D>(ka, kbase, t2, kv_hi, lane);
        dma_v_bf16<D>(vtiles, vbase, t2, kv_hi, lane);
      }
      process_tile_bf16<D, NB>(kb2, vtiles + VT, t1, kv_hi, L, qf, qnode, s_anc, a.scale_log2, m_run, l_run, o,
                               lane);
    }
  } else {
    T* vt = reinterpret_cast<T*>(s_work + (size_t)wave * D * VTS * ES);
    // float32: registers hold one tile; V is transposed through LDS by the VALU
    for (int t0 = t_first; t0 < kv_hi; t0 += t_step) {
      if (t0 != t_first) load_tile<T, D>(ta, kbase, vbase, t0, kv_hi, lane);
      process_tile<T, D, NB>(ta, t0, kv_hi, L, vt, qf, qnode, s_anc, a.scale_log2, m_run, l_run, o, lane);
    }
  }

#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    l_run[nb] += __shfl_xor(l_run[nb], 16, 64);
    l_run[nb] += __shfl_xor(l_run[nb], 32, 64);
  }

  // ---- workgroup partial: (O unnormalised, max, sum) per row ----
  const int bgr = (b * a.n_kv_heads + g) * a.n_rowblk + rb;
  const size_t pbase = ((size_t)bgr * a.nsplit + split) * a.rows_per_wg;
  if (a.wk == 1) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int rl = wr * RB + 16 * nb + lr;
#pragma unroll
      for (int db = 0; db < DB; ++db) st_dev4(a.part_o + (pbase + rl) * D + 16 * db + 4 * lg, o[db][nb]);
      if (lg == 0) {
        st_dev(a.part_m + pbase + rl, m_run[nb]);
        st_dev(a.part_l + pbase + rl, l_run[nb]);
      }
    }
  } else {
    __syncthreads();  // every wave is done with its V^T tile
    float* mo = reinterpret_cast<float*>(s_work);  // [nwaves][RB][D]
    float* mm = mo + (size_t)nwaves * RB * D;     // [nwaves][RB]   then weights
    float* ml = mm + nwaves * RB;                 // [nwaves][RB]
    float* mL = ml + nwaves * RB;                 // [wr][RB] merged sums
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int rr = 16 * nb + lr;
#pragma unroll
      for (int db = 0; db < DB; ++db)
        *reinterpret_cast<f32x4*>(mo + ((size_t)wave * RB + rr) * D + 16 * db + 4 * lg) = o[db][nb];
      if (lg == 0) {
        mm[wave * RB + rr] = m_run[nb];
        ml[wave * RB + rr] = l_run[nb];
      }
    }
    __syncthreads();
    // per row: max over the wk waves of its row group, weights 2^(m_k - M), merged sum
    for (int rl = threadIdx.x; rl < a.rows_per_wg; rl += blockDim.x) {
      const int gr = rl / RB, rr = rl - gr * RB;
      float M = kNegInf;
      for (int k = 0; k < a.wk; ++k) M = fmaxf(M, mm[(gr + a.wr * k) * RB + rr]);
      float Ls = 0.f;
      for (int k = 0; k < a.wk; ++k) {
        const int wv = gr + a.wr * k;
        const float wgt = M == kNegInf ? 0.f : __builtin_amdgcn_exp2f(mm[wv * RB + rr] - M);
        Ls += ml[wv * RB + rr] * wgt;
        mm[wv * RB + rr] = wgt;
      }
      mL[rl] = Ls;
      st_dev(a.part_m + pbase + rl, M);
      st_dev(a.part_l + pbase + rl, Ls);
    }
    __syncthreads();
    constexpr int D4 = D / 4;
    for (int idx = threadIdx.x; idx < a.rows_per_wg * D4; idx += blockDim.x) {
      const int rl = idx / D4, d = (idx - rl * D4) * 4;
      const int gr = rl / RB, rr = rl - gr * RB;
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      for (int k = 0; k < a.wk; ++k) {
        const int wv = gr + a.wr * k;
        acc += *reinterpret_cast<const f32x4*>(mo + ((size_t)wv * RB + rr) * D + d) * mm[wv * RB + rr];
      }
      st_dev4(a.part_o + (pbase + rl) * D + d, acc);
    }
  }

  // ---- completion ticket; the last split merges ----
  stores_done();
  __syncthreads();
  if (threadIdx.x == 0) *s_ticket = atomicAdd(a.counter + bgr, 1);
  __syncthreads();
  if (*s_ticket != a.nsplit - 1) return;
  if (threadIdx.x == 0) st_dev(a.counter + bgr, 0);

  // Final merge over splits, in row chunks whose (row, split) weights fit the work area:
  // w[r][s] = 2^(m_s - M) / sum_s' l_s' 2^(m_s' - M);  O[r][d] = sum_s w[r][s] * O_s[r][d].
  const int rows_here = min(a.rows_per_wg, R - row_wg);
  const size_t sbase = (size_t)bgr * a.nsplit * a.rows_per_wg;
  float* s_w = reinterpret_cast<float*>(s_work);
  const int work_floats = (int)((a.lds_work_bytes) / 4);
  const int rc_max = max(1, min(rows_here, work_floats / (2 * a.nsplit)));
  for (int r0 = 0; r0 < rows_here; r0 += rc_max) {
    const int rc = min(rc_max, rows_here - r0);
    __syncthreads();
    float* s_l = s_w + rc * a.nsplit;
    for (int idx = threadIdx.x; idx < rc * a.nsplit; idx += blockDim.x) {
      const int r = idx / a.nsplit, sp = idx - r * a.nsplit;
      const size_t pr = sbase + (size_t)sp * a.rows_per_wg + r0 + r;
      s_w[idx] = ld_dev(a.part_m + pr);
      s_l[idx] = ld_dev(a.part_l + pr);
    }
    __syncthreads();
    for (int r = threadIdx.x; r < rc; r += blockDim.x) {
      float M = kNegInf;
      for (int sp = 0; sp < a.nsplit; ++sp) M = fmaxf(M, s_w[r * a.nsplit + sp]);
      float Ls = 0.f;
      for (int sp = 0; sp < a.nsplit; ++sp) {
        const float e = __builtin_amdgcn_exp2f(s_w[r * a.nsplit + sp] - M);
        s_w[r * a.nsplit + sp] = e;
        Ls += e * s_l[r * a.nsplit + sp];
      }
      const float inv = 1.f / Ls;
      for (int sp = 0; sp < a.nsplit; ++sp) s_w[r * a.nsplit + sp] *= inv;
    }
    __syncthreads();
    constexpr int D4 = D / 4;
    constexpr int kBatch = 8;  // split partials loaded per batch, all issued before use
    for (int idx = threadIdx.x; idx < rc * D4; idx += blockDim.x) {
      const int r = idx / D4, d = (idx - r * D4) * 4;
      const float* wgt = s_w + r * a.nsplit;
      const float* po = a.part_o + (sbase + r0 + r) * D + d;
      const size_t sstride = (size_t)a.rows_per_wg * D;
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
      for (int sp0 = 0; sp0 < a.nsplit; sp0 += kBatch) {
        f32x4 buf[kBatch];
#pragma unroll
        for (int u = 0; u < kBatch; ++u)
          buf[u] = sp0 + u < a.nsplit ? ld_dev4(po + (size_t)(sp0 + u) * sstride) : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int u = 0; u < kBatch; ++u)
          if (sp0 + u < a.nsplit) acc += buf[u] * wgt[sp0 + u];
      }
      const int rr = row_wg + r0 + r;
      const int node = rr / a.group;
      const int h = g * a.group + (rr - node * a.group);
      const size_t gi = (size_t)(node0 + node) * a.hidden_size + (size_t)h * D + d;
      if (a.attn_out) *reinterpret_cast<f32x4*>(a.attn_out + gi) = acc;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float hv = Elem<T>::to_f32(a.hidden, gi + i);
        Elem<T>::store(a.x_out, gi + i, hv + acc[i]);
      }
    }
  }
}

template <typename T, int D>
static hipError_t launch_nb(int nb, dim3 grid, int threads, size_t lds, const AttnArgs& a, hipStream_t s) {
  switch (nb) {
    case 1: hipLaunchKernelGGL((tree_attn_kernel<T, D, 1>), grid, dim3(threads), lds, s, a); break;
    case 2: hipLaunchKernelGGL((tree_attn_kernel<T, D, 2>), grid, dim3(threads), lds, s, a); break;
    case 3: hipLaunchKernelGGL((tree_attn_kernel<T, D, 3>), grid, dim3(threads), lds, s, a); break;
    case 4: hipLaunchKernelGGL((tree_attn_kernel<T, D, 4>), grid, dim3(threads), lds, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename T, int D>
static hipError_t set_lds_nb(int nb, size_t lds) {
  const void* f = nullptr;
  switch (nb) {
    case 1: f = reinterpret_cast<const void*>(&tree_attn_kernel<T, D, 1>); break;
    case 2: f = reinterpret_cast<const void*>(&tree_attn_kernel<T, D, 2>); break;
    case 3: f = reinterpret_cast<const void*>(&tree_attn_kernel<T, D, 3>); break;
    case 4: f = reinterpret_cast<const void*>(&tree_attn_kernel<T, D, 4>); break;
    default: return hipErrorInvalidValue;
  }
  return hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
}

hipError_t launch_tree_attn(int dtype, int head_dim, int nb, dim3 grid, int threads, size_t lds,
                            const AttnArgs& a, hipStream_t s) {
  if (dtype == 1 && head_dim == 128) return launch_nb<bf16_t, 128>(nb, grid, threads, lds, a, s);
  if (dtype == 1 && head_dim == 64) return launch_nb<bf16_t, 64>(nb, grid, threads, lds, a, s);
  if (dtype == 0 && head_dim == 128) return launch_nb<float, 128>(nb, grid, threads, lds, a, s);
  if (dtype == 0 && head_dim == 64) return launch_nb<float, 64>(nb, grid, threads, lds, a, s);
  return hipErrorInvalidValue;
}

hipError_t set_tree_attn_lds_limit(int dtype, int head_dim, int nb, size_t lds) {
  if (dtype == 1 && head_dim == 128) return set_lds_nb<bf16_t, 128>(nb, lds);
  if (dtype == 1 && head_dim == 64) return set_lds_nb<bf16_t, 64>(nb, lds);
  if (dtype == 0 && head_dim == 128) return set_lds_nb<float, 128>(nb, lds);
  if (dtype == 0 && head_dim == 64) return set_lds_nb<float, 64>(nb, lds);
  return hipErrorInvalidValue;
}

}  // namespace respec
