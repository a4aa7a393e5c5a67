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
//   - each wave keeps two KV tiles in flight while it processes a third (with
//     several waves of rows per KV head, bf16: the waves instead share KV
//     tiles that a DMA ring brings into LDS, several tiles per barrier; see
//     the shared-tile variant below);
//   - waves of a row group are merged in LDS; each workgroup writes an
//     unnormalised partial (O, max, sum) per row;
//   - a second, wide kernel merges the splits of every row and writes O and
//     x = round(h + O) (one workgroup alone cannot pull the partials of a
//     head fast enough: a single CU's memory parallelism caps it at tens of
//     GB/s).
#include "common.hpp"
#include "kernels.hpp"

namespace respec {

// Headroom of the lazily raised softmax reference maximum (log2 units).
constexpr float kLazyMargin = 8.f;

// Bit ai of a 128-bit ancestor set.
__device__ __forceinline__ bool anc_has(const u32x4& w, int ai) {
  const uint32_t word = ai < 64 ? (ai < 32 ? w[0] : w[1]) : (ai < 96 ? w[2] : w[3]);
  return (word >> (ai & 31)) & 1u;
}

// Maxima as single instructions.  Scores come straight from the matrix cores,
// and fmaxf would first canonicalise each of them (one more instruction per
// score); no score is a signalling NaN, so the plain instruction gives the
// same maximum.
__device__ __forceinline__ float max3_f32(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}
__device__ __forceinline__ float max_f32(float a, float b) {
  float r;
  asm("v_max_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
// Maximum of the 8 scores a lane holds for one query row (two 16-key halves of
// a tile) and of the row's other three lane groups (lanes l ^ 16, l ^ 32,
// l ^ 48).  A swap of odd and even 16-lane rows between two copies of x leaves
// each lane's own and partner's values split over the two results, so their
// maximum is the pair's maximum in every lane; the 32-lane swap does the same
// for the halves.
__device__ __forceinline__ float row_max8(f32x4 a, f32x4 b) {
  float x = max_f32(max3_f32(a[0], a[1], a[2]), max3_f32(a[3], b[0], max3_f32(b[1], b[2], b[3])));
  const auto h = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = max_f32(__uint_as_float(h[0]), __uint_as_float(h[1]));
  const auto w = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return max_f32(__uint_as_float(w[0]), __uint_as_float(w[1]));
}

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
                                             const u32x4 (&anc)[NB], float scale_log2, float (&m_run)[NB],
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
          if (vis && ai >= 0) vis = qnode[nb] >= 0 && anc_has(anc[nb], ai);
          s[kb][nb][i] = vis ? s[kb][nb][i] : kNegInf;
        }
      }
    }
  }
  // online softmax (row max shared by the 4 lane groups of a row)
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const float tm = row_max8(s[0][nb], s[1][nb]);
    // m_run is a reference maximum: it is raised only when a score exceeds it by more
    // than kLazyMargin (so p <= 2^kLazyMargin), and the accumulators are rescaled only
    // then; while it is unset (-inf) the accumulators are zero and need no rescale.
    const float tmax = tm * scale_log2;
    const bool raise = tmax > m_run[nb] + kLazyMargin;
    const float mn = raise ? tmax : m_run[nb];
    const bool rescale = raise && m_run[nb] != kNegInf;
    const float alpha = rescale ? __builtin_amdgcn_exp2f(m_run[nb] - mn) : 1.f;
    const float mb = mn == kNegInf ? 0.f : mn;
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
    if (__any(rescale)) {
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
// bf16 path: K and V tiles are loaded into registers (16 bytes per lane); V is
// stored into a per-wave LDS tile and read back transposed with
// ds_read_b64_tr_b16.  (Staging V by LDS DMA instead would leave DMA and
// register loads in flight together, which the compiler's wait-count
// insertion treats as completing out of order: it would wait for every
// outstanding load before each tile.)
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

// V rows of one 32-row tile, 16 bytes per lane per piece: piece q of lane l
// is chunk (q*64 + l) % CPR of row (q*64 + l) / CPR (rows >= kv_hi clamped).
template <int D>
struct VTile {
  static constexpr int CPR = D * 2 / 16;           // 16-byte chunks per row
  static constexpr int kPieces = kKvTile * CPR / 64;
  u32x4 v[kPieces];
};

template <int D>
__device__ __forceinline__ void load_v_bf16(VTile<D>& t, const char* vbase, int t0, int kv_hi, int lane) {
  constexpr int CPR = VTile<D>::CPR;
#pragma unroll
  for (int q = 0; q < VTile<D>::kPieces; ++q) {
    const int idx = q * 64 + lane;
    const int p = min(t0 + idx / CPR, kv_hi - 1);
    t.v[q] = ld16(vbase + (size_t)p * D * 2 + (size_t)(idx % CPR) * 16);
  }
}

// Store a V tile row-major into the wave's LDS tile, chunk c of row r at
// chunk position c ^ vswz(r).
template <int D>
__device__ __forceinline__ void store_v_bf16(const VTile<D>& t, unsigned char* vtile, int lane) {
  constexpr int CPR = VTile<D>::CPR;
#pragma unroll
  for (int q = 0; q < VTile<D>::kPieces; ++q) {
    const int idx = q * 64 + lane;
    const int r = idx / CPR, c = idx % CPR;
    *reinterpret_cast<u32x4*>(vtile + r * (D * 2) + (c ^ vswz<D>(r)) * 16) = t.v[q];
  }
}

// S^T = K Q^T of one tile, unscaled: lane holds S[query 16*nb + lr][kv t0 + 16*kb + 4*lg + i].
template <int D, int NB>
__device__ __forceinline__ void scores_bf16(const KTile<D>& t, const u32x4 (&qf)[NB][D * 2 / 64], f32x4 (&s)[2][NB]) {
  constexpr int KCH = D * 2 / 64;
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
}

// V^T fragments of one LDS tile: vf[db] is the A operand of O^T += V^T P^T for
// output rows 16*db .. 16*db+15 (transposing reads, layout described above).
template <int D>
__device__ __forceinline__ void read_vt_bf16(const unsigned char* vtile, int lane, u32x4 (&vf)[D / 16]) {
  constexpr int DB = D / 16;
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
  typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
  const int lr = lane & 15, lg = lane >> 4;
  const int r = 4 * lg + lr / 4;  // row for kb = 0; kb = 1 adds 16 rows (same swizzle)
  const int sw = vswz<D>(r);
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    const int col = 16 * db + 4 * (lr % 4);
    const unsigned char* addr = vtile + r * (D * 2) + ((col >> 3) ^ sw) * 16 + (col & 7) * 2;
    const u32x2 h0 = __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(addr)));
    const u32x2 h1 =
        __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(addr + 16 * D * 2)));
    vf[db] = u32x4{h0.x, h0.y, h1.x, h1.y};
  }
}

// Tree / range mask and online softmax of one tile whose scores are in s; the
// accumulators are rescaled when the reference maximum rises, and the
// probabilities come back as the hi + lo bf16 parts of the P^T fragments.
template <int D, int NB>
__device__ __forceinline__ void softmax_p_bf16(f32x4 (&s)[2][NB], int t0, int kv_hi, int L, const int (&qnode)[NB],
                                               const u32x4 (&anc)[NB], float scale_log2, float (&m_run)[NB],
                                               float (&l_run)[NB], f32x4 (&o)[D / 16][NB], int lane,
                                               u32x4 (&phi)[NB], u32x4 (&plo)[NB], int nbc = NB) {
  constexpr int DB = D / 16;
  const int lg = lane >> 4;
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
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
          if (vis && ai >= 0) vis = qnode[nb] >= 0 && anc_has(anc[nb], ai);
          s[kb][nb][i] = vis ? s[kb][nb][i] : kNegInf;
        }
      }
    }
  }
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    if (nb >= nbc) break;  // row blocks past nbc hold no live row (wave-uniform)
    const float tm = row_max8(s[0][nb], s[1][nb]);
    // m_run is a reference maximum: it is raised only when a score exceeds it by more
    // than kLazyMargin (so p <= 2^kLazyMargin), and the accumulators are rescaled only
    // then; while it is unset (-inf) the accumulators are zero and need no rescale.
    const float tmax = tm * scale_log2;
    const bool raise = tmax > m_run[nb] + kLazyMargin;
    const float mn = raise ? tmax : m_run[nb];
    const bool rescale = raise && m_run[nb] != kNegInf;
    const float alpha = rescale ? __builtin_amdgcn_exp2f(m_run[nb] - mn) : 1.f;
    const float mb = mn == kNegInf ? 0.f : mn;
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
    if (__any(rescale)) {
#pragma unroll
      for (int db = 0; db < DB; ++db) o[db][nb] *= alpha;
    }
  }
  // P^T fragments, hi + lo bf16 parts
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    if (nb >= nbc) break;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float p0 = s[j >> 1][nb][2 * (j & 1)], p1 = s[j >> 1][nb][2 * (j & 1) + 1];
      const uint32_t h = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{p0, p1}, bf16x2));
      const float r0 = p0 - __uint_as_float(h << 16), r1 = p1 - __uint_as_float(h & 0xFFFF0000u);
      phi[nb][j] = h;
      plo[nb][j] = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{r0, r1}, bf16x2));
    }
  }
}

// O^T += V^T P^T for the output blocks db0 .. db0 + N - 1 (vf[j] holds block db0 + j).
template <int D, int NB, int N>
__device__ __forceinline__ void pv_bf16(const u32x4 (&vf)[N], int db0, const u32x4 (&phi)[NB],
                                        const u32x4 (&plo)[NB], f32x4 (&o)[D / 16][NB], int nbc = NB) {
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    if (nb >= nbc) break;  // row blocks past nbc hold no live row (wave-uniform)
#pragma unroll
    for (int j = 0; j < N; ++j) {
      o[db0 + j][nb] = mma_k64(bf16_t{}, vf[j], phi[nb], o[db0 + j][nb]);
      o[db0 + j][nb] = mma_k64(bf16_t{}, vf[j], plo[nb], o[db0 + j][nb]);
    }
  }
}

// Mask, online softmax and O^T += V^T P^T for one tile whose scores are in s
// and whose V^T fragments are in vf.
template <int D, int NB>
__device__ __forceinline__ void softmax_pv_bf16(f32x4 (&s)[2][NB], const u32x4 (&vf)[D / 16], int t0, int kv_hi,
                                                int L, const int (&qnode)[NB], const u32x4 (&anc)[NB],
                                                float scale_log2, float (&m_run)[NB], float (&l_run)[NB],
                                                f32x4 (&o)[D / 16][NB], int lane) {
  u32x4 phi[NB], plo[NB];
  softmax_p_bf16<D, NB>(s, t0, kv_hi, L, qnode, anc, scale_log2, m_run, l_run, o, lane, phi, plo);
  pv_bf16<D, NB, D / 16>(vf, 0, phi, plo, o);
}

// Ancestor-or-self bitsets of each lane's query nodes, walked up the parent
// array held in registers (lane l holds parent[l] and parent[l + 64]); all
// lanes take part in every exchange and the walk ends when every lane has
// reached the root or an invalid parent (parents must strictly decrease).
template <int NB>
__device__ __forceinline__ void ancestor_bits(const int (&qnode)[NB], int p_lo, int p_hi, int n_nodes,
                                              u32x4 (&anc)[NB]) {
  // Take the parents out of the loads' bookkeeping here, in straight-line
  // code: the compiler then waits for these two loads only, not (as it does
  // for loaded values used in a load-free loop) for every load in flight.
  asm volatile("" : "+v"(p_lo), "+v"(p_hi));
  const int lane = (int)(threadIdx.x & 63);
  p_lo = lane < n_nodes ? p_lo : -1;
  p_hi = lane + 64 < n_nodes ? p_hi : -1;
  int x[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    x[nb] = qnode[nb];
    anc[nb] = u32x4{0u, 0u, 0u, 0u};
  }
  const bool two = n_nodes > 64;  // (uniform) parents of nodes 64.. are needed
  for (int step = 0; step < kMaxNodes; ++step) {
    bool any = false;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int xv = x[nb];
      const uint32_t bit = xv >= 0 ? 1u << (xv & 31) : 0u;
      const int w = xv >> 5;
      anc[nb][0] |= w == 0 ? bit : 0u;
      anc[nb][1] |= w == 1 ? bit : 0u;
      anc[nb][2] |= w == 2 ? bit : 0u;
      anc[nb][3] |= w == 3 ? bit : 0u;
      const int sel = (xv & 63) << 2;
      int p = __builtin_amdgcn_ds_bpermute(sel, p_lo);
      if (two) {
        const int ph = __builtin_amdgcn_ds_bpermute(sel, p_hi);
        p = xv >= 64 ? ph : p;
      }
      x[nb] = (xv > 0 && p >= 0 && p < xv) ? p : -1;
      any |= x[nb] >= 0;
    }
    if (!__any(any)) break;
  }
}

// The workgroup's unnormalised partial (O, reference max m, sum l) of each of its
// rows, from the waves' accumulators (after the row-wide sum of l).  With one
// wave per row group it is stored directly; otherwise the wk waves of a row group
// combine their (O, m, l) through LDS (s_work, LDS no longer read by any wave).
template <int D, int NB>
__device__ __forceinline__ void store_partial(const AttnArgs& a, unsigned char* s_work, const f32x4 (&o)[D / 16][NB],
                                              const float (&m_run)[NB], const float (&l_run)[NB], size_t pbase,
                                              int wave, int nwaves, int lane) {
  constexpr int DB = D / 16;
  constexpr int RB = 16 * NB;
  const int lr = lane & 15, lg = lane >> 4;
  const int wr = wave % a.wr, wk = wave / a.wr;
  if (a.wk == 1) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const int rl = wr * RB + 16 * nb + lr;
#pragma unroll
      for (int db = 0; db < DB; ++db)
        *reinterpret_cast<f32x4*>(a.part_o + (pbase + rl) * D + 16 * db + 4 * lg) = o[db][nb];
      if (lg == 0) {
        a.part_m[pbase + rl] = m_run[nb];
        a.part_l[pbase + rl] = l_run[nb];
      }
    }
  } else {
    // The wk waves of a row group combine their (O, m, l) through LDS.  Every wave
    // stores its accumulators lane-major (so[wave][db][nb][lane], 16 bytes per lane:
    // consecutive lanes write consecutive addresses, no bank conflicts), then each wave
    // of the group combines the output blocks db = wk, wk + a.wk, ... of the group's
    // rows in registers, lane by lane (every wave holds row lr + 16 nb, columns
    // 16 db + 4 lg + i, in the same lane):
    //   M = max_k m_k,  w_k = 2^(m_k - M),  l = sum_k w_k l_k,  O = sum_k w_k O_k.
    __syncthreads();  // every wave is done with its V tiles
    f32x4* so = reinterpret_cast<f32x4*>(s_work);                       // [nwaves][DB][NB][64]
    float* sm = reinterpret_cast<float*>(so + (size_t)nwaves * DB * NB * 64);  // [nwaves][NB][64]
    float* sl = sm + nwaves * NB * 64;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
      for (int db = 0; db < DB; ++db) so[((wave * DB + db) * NB + nb) * 64 + lane] = o[db][nb];
      sm[(wave * NB + nb) * 64 + lane] = m_run[nb];
      sl[(wave * NB + nb) * 64 + lane] = l_run[nb];
    }
    __syncthreads();
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      float M = kNegInf;
      for (int k = 0; k < a.wk; ++k) M = fmaxf(M, sm[((wr + a.wr * k) * NB + nb) * 64 + lane]);
      float wgt[4], Ls = 0.f;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int wv = wr + a.wr * k;
        const float mk = k < a.wk ? sm[(wv * NB + nb) * 64 + lane] : kNegInf;
        wgt[k] = mk == kNegInf ? 0.f : __builtin_amdgcn_exp2f(mk - M);
        Ls += k < a.wk ? sl[(wv * NB + nb) * 64 + lane] * wgt[k] : 0.f;
      }
      const int rl = wr * RB + 16 * nb + lr;
      for (int db = wk; db < DB; db += a.wk) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int k = 0; k < 4; ++k)
          if (k < a.wk) acc += so[(((wr + a.wr * k) * DB + db) * NB + nb) * 64 + lane] * wgt[k];
        *reinterpret_cast<f32x4*>(a.part_o + (pbase + rl) * D + 16 * db + 4 * lg) = acc;
      }
      if (wk == 0 && lg == 0) {
        a.part_m[pbase + rl] = M;
        a.part_l[pbase + rl] = Ls;
      }
    }
  }

}

// Rows of sequence b's KV range (prefix + tree); invalid device data degrades
// to an empty sequence.  The merge computes the same, so both agree on the
// flat partition.
struct SeqRows {
  int node0, n_nodes, L;
};
__device__ __forceinline__ SeqRows seq_rows(const AttnArgs& a, int b) {
  const int node0 = a.node_off[b], node1 = a.node_off[b + 1];
  int n_nodes = node1 - node0;
  if (node0 < 0 || node1 > a.total_nodes || n_nodes < 1 || n_nodes > a.max_nodes) n_nodes = 0;
  int L = a.kv_len[b];
  L = max(0, min(L, a.kv_cap - n_nodes));
  return SeqRows{node0, n_nodes, n_nodes > 0 ? L : 0};
}

// Flat partition of a head's KV tiles over the sequences of the batch (one
// wave; lane l describes sequence l < batch <= 64): tiles of each sequence,
// their exclusive prefix and the total.
struct FlatTiles {
  int tiles, pre, total;
};
__device__ __forceinline__ FlatTiles flat_tiles(const AttnArgs& a, int lane) {
  int nt = 0;
  if (lane < a.batch) {
    const SeqRows sr = seq_rows(a, lane);
    nt = sr.n_nodes > 0 ? (sr.L + sr.n_nodes + kKvTile - 1) / kKvTile : 0;
  }
  int incl = nt;
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(incl, o, 64);
    if (lane >= o) incl += y;
  }
  return FlatTiles{nt, incl - nt, __shfl(incl, 63, 64)};
}
// The piece (of P over `total` tiles, boundaries floor(p * total / P)) that holds tile x.
__device__ __forceinline__ int flat_piece(int x, int P, int total) {
  return (int)(((long long)(x + 1) * P - 1) / total);
}

// One segment of work: KV rows [kv_lo, min(kv_hi, t_rows)) of sequence b, KV
// head g, row block rb, written to partial slot `slot`.
template <typename T, int D, int NB>
__device__ __forceinline__ void attn_segment(const AttnArgs& a, unsigned char* s_work, int b, int g, int rb,
                                             int kv_lo, int kv_hi_req, int slot) {
  constexpr int ES = Elem<T>::kBytes;
  constexpr int KCH = D * ES / 64;     // 64-byte K-chunks per head row
  constexpr int DB = D / 16;           // 16-wide output blocks along D
  constexpr int VTS = kKvTile + kVtPad;  // elements per transposed-V row (float32 path)
  constexpr int RB = 16 * NB;          // query rows per wave

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform: scalar branches below
  const int lr = lane & 15, lg = lane >> 4;
  const int nwaves = blockDim.x >> 6;
  const int wr = wave % a.wr, wk = wave / a.wr;
  const int split = slot;

  const SeqRows sr = seq_rows(a, b);
  const int node0 = sr.node0, n_nodes = sr.n_nodes, L = sr.L;
  const int R = n_nodes * a.group;
  const int row_wg = rb * a.rows_per_wg;
  if (row_wg >= R) return;  // uniform over every split of this row block

  const size_t head_row0 = ((size_t)b * a.n_kv_heads + g) * (size_t)a.kv_cap;
  const char* kbase = reinterpret_cast<const char*>(a.k_cache) + head_row0 * D * ES;
  const char* vbase = reinterpret_cast<const char*>(a.v_cache) + head_row0 * D * ES;
  const int t_rows = L + n_nodes;
  const int kv_hi = min(kv_hi_req, t_rows);
  const int t_first = kv_lo + wk * kKvTile, t_step = kKvTile * a.wk;
  const int n_tiles = t_first < kv_hi ? (kv_hi - t_first + t_step - 1) / t_step : 0;

  // Issue order (the vector-memory counter drains in order): parents, queries,
  // then the first two KV tiles.
  const int p_lo = a.parent[node0 + min(lane, n_nodes - 1)];  // parent[lane] (valid lanes)
  const int p_hi = a.parent[node0 + min(lane + 64, n_nodes - 1)];
  const int row_wave = row_wg + wr * RB;
  u32x4 qf[NB][KCH];
  int qnode[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    // rows past the group's last are loaded from the first row (issued by every lane, so
    // that every lane's loads are counted alike) and zeroed
    const int r = row_wave + 16 * nb + lr;
    const bool live = r < R;
    const int rc = live ? r : 0;
    const int node = rc / a.group;
    const int h = g * a.group + (rc - node * a.group);
    qnode[nb] = live ? node : -1;
    const char* src = reinterpret_cast<const char*>(a.hidden) +
                      ((size_t)(node0 + node) * a.hidden_size + (size_t)h * D) * ES;
#pragma unroll
    for (int kc = 0; kc < KCH; ++kc) {
      const u32x4 v = ld16(src + kc * 64 + lg * 16);
      qf[nb][kc] = live ? v : u32x4{0, 0, 0, 0};
    }
  }

  float m_run[NB], l_run[NB];
  f32x4 o[DB][NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    m_run[nb] = kNegInf;
    l_run[nb] = 0.f;
#pragma unroll
    for (int db = 0; db < DB; ++db) o[db][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  u32x4 anc[NB];

  if constexpr (ES == 2) {
    // Two tiles in flight per wave, all in registers: K fragments go straight
    // to the matrix cores; V is written to the wave's LDS tile and read back
    // transposed.  Tile i is waited for, its scores and V^T fragments taken,
    // and tile i+2 is issued into the registers it frees, so two tiles stream
    // while tile i is processed.
    unsigned char* vt = s_work + (size_t)wave * kKvTile * D * 2;
    const int t_last = max(kv_hi - 1, 0);
    auto tile_row = [&](int i) { return i < n_tiles ? t_first + i * t_step : t_last; };
    KTile<D> ka, kb;
    VTile<D> va, vb;
    // (kv_hi >= 1 always: the sequence has a node, and a split starts before its end or
    // is clipped to it; so every clamped row below is a valid cache row)
    // (scheduling barriers keep tile 0's loads ahead of tile 1's: the loop's
    // wait counts assume that order)
    // (tile 1 is requested by the first step, once tile 0's scores are taken:
    // the wave then starts on tile 0 while tile 1 streams, instead of first
    // waiting for every request to be accepted)
    load_k_bf16<D>(ka, kbase, tile_row(0), kv_hi, lane);
    load_v_bf16<D>(va, vbase, tile_row(0), kv_hi, lane);
    __builtin_amdgcn_sched_barrier(0);
    // the tree's own rows (L..) need the ancestor masks: only a split that reaches them
    // waits for the parents (uniform)
    if (kv_hi > L)
      ancestor_bits<NB>(qnode, p_lo, p_hi, n_nodes, anc);
    else
      for (int nb = 0; nb < NB; ++nb) anc[nb] = u32x4{0u, 0u, 0u, 0u};
    // one tile: scores from K, V through LDS, then the tile two ahead issued into the freed registers
    auto tile_step = [&](KTile<D>& kt, VTile<D>& vv, int i, bool refill, bool first) {
      f32x4 s[2][NB];
      scores_bf16<D, NB>(kt, qf, s);
      if (first) {
        load_k_bf16<D>(kb, kbase, tile_row(1), kv_hi, lane);
        load_v_bf16<D>(vb, vbase, tile_row(1), kv_hi, lane);
      }
      store_v_bf16<D>(vv, vt, lane);
      wave_lds_sync();
      u32x4 vf[DB];
      read_vt_bf16<D>(vt, lane, vf);
      if (refill) {
        load_k_bf16<D>(kt, kbase, tile_row(i + 2), kv_hi, lane);
        load_v_bf16<D>(vv, vbase, tile_row(i + 2), kv_hi, lane);
      }
      softmax_pv_bf16<D, NB>(s, vf, t_first + i * t_step, kv_hi, L, qnode, anc, a.scale_log2, m_run, l_run, o, lane);
      wave_lds_sync();  // this tile's V^T reads precede the next tile's writes
    };
    // Tile 0, then the steady state from tile 1: both halves refill real
    // tiles, so the count of loads behind every tile is the same on every
    // pass.  The last tiles (straight-line code) refill only while tiles
    // remain: no load is left in flight for the workgroup's merge barrier to
    // wait for.
    // A wave with at most two tiles (short splits) requests the second one at
    // once: it then waits for one memory latency instead of two in a row.
    // (Past the last tile the request repeats the last row: cached, unused.)
    if (n_tiles <= 2) {
      load_k_bf16<D>(kb, kbase, tile_row(1), kv_hi, lane);
      load_v_bf16<D>(vb, vbase, tile_row(1), kv_hi, lane);
      if (n_tiles > 0) tile_step(ka, va, 0, false, false);
      if (n_tiles > 1) tile_step(kb, vb, 1, false, false);
    } else {
    int i = 1;
    tile_step(ka, va, 0, 2 < n_tiles, true);
    for (; i + 4 <= n_tiles; i += 2) {
      tile_step(kb, vb, i, true, false);
      tile_step(ka, va, i + 1, true, false);
    }
    if (i < n_tiles) tile_step(kb, vb, i, i + 2 < n_tiles, false);
    if (i + 1 < n_tiles) tile_step(ka, va, i + 1, i + 3 < n_tiles, false);
    if (i + 2 < n_tiles) tile_step(kb, vb, i + 2, false, false);
    }
  } else {
    // float32: registers hold one tile; V is transposed through LDS by the VALU
    if (kv_hi > L)
      ancestor_bits<NB>(qnode, p_lo, p_hi, n_nodes, anc);
    else
      for (int nb = 0; nb < NB; ++nb) anc[nb] = u32x4{0u, 0u, 0u, 0u};
    T* vt = reinterpret_cast<T*>(s_work + (size_t)wave * D * VTS * ES);
    AttnTile<T, D> ta;
    for (int i = 0; i < n_tiles; ++i) {
      const int t0 = t_first + i * t_step;
      load_tile<T, D>(ta, kbase, vbase, t0, kv_hi, lane);
      process_tile<T, D, NB>(ta, t0, kv_hi, L, vt, qf, qnode, anc, a.scale_log2, m_run, l_run, o, lane);
    }
  }

#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    l_run[nb] += xchg<4>(l_run[nb]);
    l_run[nb] += xchg<5>(l_run[nb]);
  }

  // ---- workgroup partial: (O unnormalised, max, sum) per row ----
  const int bgr = (b * a.n_kv_heads + g) * a.n_rowblk + rb;
  const size_t pbase = ((size_t)bgr * a.nsplit + split) * a.rows_per_wg;
  store_partial<D, NB>(a, s_work, o, m_run, l_run, pbase, wave, nwaves, lane);
}

template <typename T, int D, int NB, bool Flat>
__global__ __launch_bounds__(256) void tree_attn_kernel(AttnArgs a) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int g = blockIdx.y / a.n_rowblk, rb = blockIdx.y % a.n_rowblk;
  if constexpr (!Flat) {
    attn_segment<T, D, NB>(a, smem, blockIdx.z, g, rb, blockIdx.x * a.chunk, blockIdx.x * a.chunk + a.chunk,
                           blockIdx.x);
    return;
  }
  // Flat partition (ragged batches): piece p of this head's tiles over every
  // sequence, so that every workgroup streams the same number of KV tiles
  // whatever the lengths; a piece runs one segment per sequence it touches.
  const int lane = threadIdx.x & 63;
  const FlatTiles ft = flat_tiles(a, lane);
  const int P = a.flat, p = blockIdx.x;
  if (ft.total == 0) return;
  const int T0 = (int)((long long)p * ft.total / P), T1 = (int)((long long)(p + 1) * ft.total / P);
  const bool touches = lane < a.batch && ft.tiles > 0 && ft.pre < T1 && ft.pre + ft.tiles > T0;
  uint64_t seqs = __ballot(touches);
  bool first = true;
  while (seqs) {
    const int b = __builtin_ctzll(seqs);
    seqs &= seqs - 1;
    const int pre = __shfl(ft.pre, b, 64), nt = __shfl(ft.tiles, b, 64);
    const int lo = max(T0, pre) - pre, hi = min(T1, pre + nt) - pre;
    const int slot = p - flat_piece(pre, P, ft.total);
    if (!first) __syncthreads();  // the previous segment's merge is done with the LDS
    first = false;
    attn_segment<T, D, NB>(a, smem, b, g, rb, lo * kKvTile, hi * kKvTile, slot);
  }
}

// ---------------------------------------------------------------------------
// Shared-tile variant (bf16; a KV head's query rows span 2-8 waves).  Every
// wave of such a workgroup needs the same KV rows, so each KV tile is fetched
// once per workgroup, straight into LDS by DMA (global_load_lds, 16 bytes per
// lane), into a ring of S slots:
//   - wave 0 requests the K half and wave 1 the V half of every tile;
//   - a pass consumes TP = KG*TPG tiles (each of the KG key groups takes TPG
//     of them, in tile order) while the next S-TP are in flight: a requesting
//     wave waits until only its S-2*TP newest tiles are pending, then one
//     barrier publishes the pass's tiles to every wave and, as every wave has
//     finished the previous pass by then, frees that pass's slots for the
//     tiles S ahead, requested right after.  Several tiles per pass (one
//     barrier for all of them) let the waves of a SIMD drift apart within the
//     pass instead of meeting at every tile;
//   - the DMA requests are inline assembly (see dma_half_asm), so the K
//     fragments (A operand of S^T = K Q^T) and the transposed V fragments are
//     ordinary LDS reads that the compiler schedules; the barrier's own waits
//     order them against the ring;
//   - each wave owns 16*NB query rows of its own: no cross-wave merge.
// K slot layout: 32 rows x D bf16, chunk c of row r at chunk position
// c ^ kswz(r), so that a quarter-wave reading one chunk column of 16 rows hits
// 64 distinct banks; V slots use the layout of the register path (vswz).
template <int D>
__device__ __forceinline__ int kswz(int r) {
  return D == 128 ? (r & 15) : ((r >> 1) & 7);
}

// Request one half (K or V) of a 32-row tile into an LDS slot, 16 bytes per
// lane (global_load_lds_dwordx4); rows at or past kv_hi are clamped to
// kv_hi - 1 (masked, or weighted by zero, as above).  Issued as inline
// assembly so that the compiler does not see an LDS write in flight: it then
// schedules the ring's LDS reads freely (instead of waiting for every
// outstanding request before each of them), and the kernel's own waits order
// them.  The tile base is uniform (scalar registers), each lane adds a 32-bit
// offset; M0 holds the LDS destination (saved and restored around the
// request) and needs one wait state before the request.
// Per-lane source offsets of a half-tile, one per DMA instruction (rows past
// kv_hi clamped when the tile is not whole).  A whole tile's offsets do not
// depend on the tile, so a requesting wave computes them once (DmaOffsets).
template <int D, bool V>
struct DmaLayout {
  static constexpr int CPR = D * 2 / 16;  // 16-byte chunks per row
  static constexpr int RPI = 64 / CPR;    // rows per DMA instruction (1 KB)
  static constexpr int N = kKvTile / RPI;
  __device__ __forceinline__ static uint32_t at(int q, int lane, int t0, int kv_hi, bool full) {
    const int r = q * RPI + lane / CPR, pos = lane % CPR;
    const int c = pos ^ (V ? vswz<D>(r) : kswz<D>(r));  // chunk that belongs at position pos
    const int rr = full ? r : min(t0 + r, kv_hi - 1) - t0;  // rows past kv_hi: row kv_hi - 1 (t0 <= kv_hi - 1)
    return (uint32_t)(rr * D * 2 + c * 16);
  }
};
template <int D>
struct DmaOffsets {
  uint32_t off[DmaLayout<D, false>::N];
  __device__ __forceinline__ void init(bool v_half, int lane) {  // v_half uniform
#pragma unroll
    for (int q = 0; q < DmaLayout<D, false>::N; ++q)
      off[q] = v_half ? DmaLayout<D, true>::at(q, lane, 0, kKvTile, true) : DmaLayout<D, false>::at(q, lane, 0, kKvTile, true);
  }
};

template <int D, bool V>
__device__ __forceinline__ void dma_half_asm(uint32_t lds_dst, const char* base, int t0, int kv_hi, int lane,
                                             const DmaOffsets<D>& pre) {
  using O = DmaLayout<D, V>;
  // the tile base and the LDS destination are uniform: made scalar explicitly for the asm operands
  const uint64_t tb_u = reinterpret_cast<uint64_t>(base + (size_t)t0 * D * 2);
  const uint64_t tb = ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(tb_u >> 32)) << 32) |
                      (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)tb_u);
  lds_dst = __builtin_amdgcn_readfirstlane(lds_dst);
  auto request = [&](int q, uint32_t off) {
    uint32_t saved;
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %1\n\t"
        "s_nop 0\n\t"
        "global_load_lds_dwordx4 %2, %3\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "s"(lds_dst + q * 1024), "v"(off), "s"(tb)
        : "memory");
  };
  if (t0 + kKvTile <= kv_hi) {  // (uniform) a whole tile: the precomputed offsets
#pragma unroll
    for (int q = 0; q < O::N; ++q) request(q, pre.off[q]);
  } else {
#pragma unroll
    for (int q = 0; q < O::N; ++q) request(q, O::at(q, lane, t0, kv_hi, false));
  }
}

template <int D, int NB, int S, int KG, int TPG>
__global__ __launch_bounds__(512) void tree_attn_shared_kernel(AttnArgs a) {
  constexpr int KCH = D * 2 / 64;
  constexpr int DB = D / 16;
  constexpr int RB = 16 * NB;
  constexpr int kTile = kKvTile * D * 2;  // bytes of one K or V half-tile
  constexpr int kStage = 2 * kTile;
  constexpr int kLpt = kTile / 1024;      // DMA instructions per half-tile
  constexpr int TP = KG * TPG;            // tiles per pass
  static_assert(S > 2 * TP && (S - 2 * TP) * kLpt <= 63, "vmcnt holds at most 63 pending requests");

  extern __shared__ __align__(16) unsigned char smem[];
  const uint32_t lds0 = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) unsigned char*)smem;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  // Roles: key group grp, row wave rw.  Waves w and w + 4 share a SIMD.  With two key groups
  // the last row wave of each group holds the fewest live rows (65 rows: blocks 2, 2 and 1),
  // so those two roles go to waves 0 and 1, whose SIMDs also carry waves 4 and 5: no SIMD then
  // holds two full row waves of a three-wave group (65 rows: at most 3 blocks per SIMD, not 4).
  int grp = 0, rw = wave;
  if constexpr (KG > 1) {
    if (a.wr == 1) {
      grp = wave;
      rw = 0;
    } else if (wave < 2) {
      grp = wave;
      rw = a.wr - 1;
    } else {
      const int j = wave - 2;
      grp = j / (a.wr - 1);
      rw = j - grp * (a.wr - 1);
    }
    grp = __builtin_amdgcn_readfirstlane(grp);
    rw = __builtin_amdgcn_readfirstlane(rw);
  }
  const int lr = lane & 15, lg = lane >> 4;
  const int b = blockIdx.z;
  const int g = blockIdx.y / a.n_rowblk, rb = blockIdx.y % a.n_rowblk;
  const int split = blockIdx.x;

  const int node0 = a.node_off[b], node1 = a.node_off[b + 1];
  int n_nodes = node1 - node0;
  if (node0 < 0 || node1 > a.total_nodes || n_nodes < 1 || n_nodes > a.max_nodes) n_nodes = 0;
  int L = a.kv_len[b];
  L = max(0, min(L, a.kv_cap - n_nodes));
  const int R = n_nodes * a.group;
  const int row_wg = rb * a.rows_per_wg;
  if (row_wg >= R) return;  // uniform over the workgroup

  const size_t head_row0 = ((size_t)b * a.n_kv_heads + g) * (size_t)a.kv_cap;
  const char* kbase = reinterpret_cast<const char*>(a.k_cache) + head_row0 * D * 2;
  const char* vbase = reinterpret_cast<const char*>(a.v_cache) + head_row0 * D * 2;
  const int t_rows = L + n_nodes;
  const int kv_lo = split * a.chunk;
  const int kv_hi = min(kv_lo + a.chunk, t_rows);
  const int n_tiles = kv_lo < kv_hi ? (kv_hi - kv_lo + kKvTile - 1) / kKvTile : 0;
  const int t_last = max(kv_hi - 1, 0);
  auto tile_row = [&](int i) { return i < n_tiles ? kv_lo + i * kKvTile : t_last; };

  int p_lo = a.parent[node0 + min(lane, n_nodes - 1)];
  int p_hi = a.parent[node0 + min(lane + 64, n_nodes - 1)];
  const int row_wave = row_wg + rw * RB;
  u32x4 qf[NB][KCH];
  int qnode[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int r = row_wave + 16 * nb + lr;
    const bool live = r < R;
    const int rc = live ? r : 0;
    const int node = rc / a.group;
    const int h = g * a.group + (rc - node * a.group);
    qnode[nb] = live ? node : -1;
    const char* src = reinterpret_cast<const char*>(a.hidden) +
                      ((size_t)(node0 + node) * a.hidden_size + (size_t)h * D) * 2;
#pragma unroll
    for (int kc = 0; kc < KCH; ++kc) {
      const u32x4 v = ld16(src + kc * 64 + lg * 16);
      qf[nb][kc] = live ? v : u32x4{0, 0, 0, 0};
    }
  }

  // Every wave has its parents and queries before the first requests are
  // issued: the compiler's wait counts do not see the requests, so a value
  // loaded before them and used after them would be waited for behind every
  // request in flight (and the wait is shared by the waves that issue none).
  asm volatile("" : "+v"(p_lo), "+v"(p_hi));
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int kc = 0; kc < KCH; ++kc) asm volatile("" : "+v"(qf[nb][kc]));
  // the first S - TP tiles (kv_hi >= 1, so every clamped row is a valid cache row)
  DmaOffsets<D> doff;  // wave 0: K halves, wave 1: V halves
  if (wave < 2) doff.init(wave == 1, lane);
  if (wave < 2) {
#pragma unroll
    for (int st = 0; st < S - TP; ++st) {
      if (wave == 0)
        dma_half_asm<D, false>(lds0 + st * kStage, kbase, tile_row(st), kv_hi, lane, doff);
      else
        dma_half_asm<D, true>(lds0 + st * kStage + kTile, vbase, tile_row(st), kv_hi, lane, doff);
    }
  }

  float m_run[NB], l_run[NB];
  f32x4 o[DB][NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    m_run[nb] = kNegInf;
    l_run[nb] = 0.f;
#pragma unroll
    for (int db = 0; db < DB; ++db) o[db][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  u32x4 anc[NB];
  if (kv_hi > L)  // (uniform) only a split that reaches the tree's own rows needs the masks
    ancestor_bits<NB>(qnode, p_lo, p_hi, n_nodes, anc);
  else
    for (int nb = 0; nb < NB; ++nb) anc[nb] = u32x4{0u, 0u, 0u, 0u};
  // row blocks of this wave that hold a live row (blocks past the group's last row are skipped)
  const int nbc = __builtin_amdgcn_readfirstlane(min(NB, max(0, (R - row_wave + 15) / 16)));

  // Pass j consumes tiles TP*j .. TP*j+TP-1 (group q takes tiles TP*j + KG*r + q,
  // r < TPG) from slots s0 .. s0+TP-1 (mod S); the slots of the previous pass's
  // tiles are refilled with the tiles S ahead of them.
  int s0 = 0;  // ring slot of tile TP*j
  for (int j = 0; TP * j < n_tiles; ++j) {
    // tiles TP*j .. TP*j+TP-1 have landed (a requesting wave waits for its own
    // requests) and every wave's reads of the previous pass are done: one
    // barrier covers both
    if (wave < 2)
      asm volatile("s_waitcnt vmcnt(%0)\n\ts_waitcnt lgkmcnt(0)\n\ts_barrier" ::"n"((S - 2 * TP) * kLpt) : "memory");
    else
      asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    if (wave < 2) {
#pragma unroll
      for (int q = 0; q < TP; ++q) {
        int sl = s0 - TP + q;
        sl = sl < 0 ? sl + S : sl;
        const int t_new = TP * j - TP + q + S;
        if (wave == 0)
          dma_half_asm<D, false>(lds0 + sl * kStage, kbase, tile_row(t_new), kv_hi, lane, doff);
        else
          dma_half_asm<D, true>(lds0 + sl * kStage + kTile, vbase, tile_row(t_new), kv_hi, lane, doff);
      }
    }
#pragma unroll
    for (int r = 0; r < TPG; ++r) {
    const int t = TP * j + KG * r + grp;
    if (t < n_tiles) {
      int slot = s0 + KG * r + grp;
      slot = slot >= S ? slot - S : slot;
      const unsigned char* kt = smem + slot * kStage;
      KTile<D> kf;
      {
        const int sw = kswz<D>(lr);  // kswz(16 + lr) == kswz(lr)
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int kc = 0; kc < KCH; ++kc)
            kf.k[kb][kc] = *reinterpret_cast<const u32x4*>(kt + (16 * kb + lr) * D * 2 + (((4 * kc + lg) ^ sw) << 4));
      }
      f32x4 s[2][NB];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          if (nb >= nbc) break;
          f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
          for (int kc = 0; kc < KCH; ++kc) acc = mma_k64(bf16_t{}, kf.k[kb][kc], qf[nb][kc], acc);
          s[kb][nb] = acc;
        }
      u32x4 vf[DB];
      read_vt_bf16<D>(kt + kTile, lane, vf);
      u32x4 phi[NB], plo[NB];
      softmax_p_bf16<D, NB>(s, kv_lo + t * kKvTile, kv_hi, L, qnode, anc, a.scale_log2, m_run, l_run, o, lane, phi,
                            plo, nbc);
      pv_bf16<D, NB, DB>(vf, 0, phi, plo, o, nbc);
    }
    }
    s0 += TP;
    s0 = s0 >= S ? s0 - S : s0;
  }
  // the DMAs past the last tile must land before the workgroup's LDS is released
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");

#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    l_run[nb] += xchg<4>(l_run[nb]);
    l_run[nb] += xchg<5>(l_run[nb]);
  }
  if constexpr (KG > 1) {
    // Key group 1 hands its (max, sum, O) to group 0 through the ring's LDS,
    // lane by lane (both hold the same rows in the same lanes):
    //   M = max(m0, m1),  w_q = 2^(m_q - M),  l = w0 l0 + w1 l1,  O = w0 O0 + w1 O1.
    constexpr int kX = DB * NB * 4 + 2 * NB;  // floats per lane
    __syncthreads();  // every wave is done with the ring
    float* xo = reinterpret_cast<float*>(smem) + (size_t)rw * kX * 64 + lane;
    if (grp == 1) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int i = 0; i < 4; ++i) xo[((nb * DB + db) * 4 + i) * 64] = o[db][nb][i];
        xo[(DB * NB * 4 + 2 * nb) * 64] = m_run[nb];
        xo[(DB * NB * 4 + 2 * nb + 1) * 64] = l_run[nb];
      }
    }
    __syncthreads();
    if (grp != 0) return;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      const float m1 = xo[(DB * NB * 4 + 2 * nb) * 64], l1 = xo[(DB * NB * 4 + 2 * nb + 1) * 64];
      const float M = fmaxf(m_run[nb], m1);
      const float w0 = m_run[nb] == kNegInf ? 0.f : __builtin_amdgcn_exp2f(m_run[nb] - M);
      const float w1 = m1 == kNegInf ? 0.f : __builtin_amdgcn_exp2f(m1 - M);
      l_run[nb] = l_run[nb] * w0 + l1 * w1;
      m_run[nb] = M;
#pragma unroll
      for (int db = 0; db < DB; ++db)
#pragma unroll
        for (int i = 0; i < 4; ++i) o[db][nb][i] = o[db][nb][i] * w0 + xo[((nb * DB + db) * 4 + i) * 64] * w1;
    }
  }
  const int bgr = (b * a.n_kv_heads + g) * a.n_rowblk + rb;
  const size_t pbase = ((size_t)bgr * a.nsplit + split) * a.rows_per_wg;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int rl = rw * RB + 16 * nb + lr;
    if (row_wg + rl >= R) continue;  // rows past the group's last are never merged
#pragma unroll
    for (int db = 0; db < DB; ++db)
      *reinterpret_cast<f32x4*>(a.part_o + (pbase + rl) * D + 16 * db + 4 * lg) = o[db][nb];
    if (lg == 0) {
      a.part_m[pbase + rl] = m_run[nb];
      a.part_l[pbase + rl] = l_run[nb];
    }
  }
}

// Split merge and residual: one workgroup per (sequence, KV head, row block,
// chunk of 256 / (D/4) rows); each thread owns one (row, 4-column) item and
// requests the partials, maxima and sums of 8 splits at a time.
//   w_s = 2^(m_s - M) / sum_s' l_s' 2^(m_s' - M),  M = max_s m_s;
//   O = sum_s w_s O_s;  x = round(h + O).
// The partials come from the attention kernel that ran before it on the same
// stream, so plain loads see them.
template <typename T, int D>
__global__ __launch_bounds__(256) void attn_merge_kernel(AttnArgs a) {
  constexpr int D4 = D / 4;
  constexpr int kRows = 256 / D4;   // rows per workgroup
  constexpr int kBatch = 8;         // splits requested per batch
  const int bgr = blockIdx.y;
  const int rb = bgr % a.n_rowblk, g = (bgr / a.n_rowblk) % a.n_kv_heads, b = bgr / (a.n_rowblk * a.n_kv_heads);
  const int node0 = a.node_off[b], node1 = a.node_off[b + 1];
  int n_nodes = node1 - node0;
  if (node0 < 0 || node1 > a.total_nodes || n_nodes < 1 || n_nodes > a.max_nodes) n_nodes = 0;
  const int R = n_nodes * a.group;
  const int row_wg = rb * a.rows_per_wg;
  const int rl = blockIdx.x * kRows + (int)threadIdx.x / D4;  // row within the row block
  const int d = ((int)threadIdx.x % D4) * 4;
  // partials of this sequence: every split, or (flat partition) the pieces its tiles span
  int nsp = a.nsplit;
  if (a.flat) {
    const FlatTiles ft = flat_tiles(a, (int)threadIdx.x & 63);
    const int pre = __shfl(ft.pre, b, 64), nt = __shfl(ft.tiles, b, 64);
    nsp = nt > 0 ? flat_piece(pre + nt - 1, a.flat, ft.total) - flat_piece(pre, a.flat, ft.total) + 1 : 0;
  }
  if (rl >= a.rows_per_wg || row_wg + rl >= R) return;
  const size_t sbase = (size_t)bgr * a.nsplit * a.rows_per_wg + rl;
  const size_t sstride = (size_t)a.rows_per_wg;

  const int rr = row_wg + rl;
  const int node = rr / a.group;
  const int h = g * a.group + (rr - node * a.group);
  const size_t gi = (size_t)(node0 + node) * a.hidden_size + (size_t)h * D + d;
  f32x4 hv;
#pragma unroll
  for (int i = 0; i < 4; ++i) hv[i] = Elem<T>::to_f32(a.hidden, gi + i);

  float M = kNegInf, Ls = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int sp0 = 0; sp0 < nsp; sp0 += kBatch) {
    float mv[kBatch], lv[kBatch];
    f32x4 ov[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const int sp = sp0 + u;
      const bool ok = sp < nsp;
      const size_t pr = sbase + (size_t)(ok ? sp : 0) * sstride;
      mv[u] = ok ? a.part_m[pr] : kNegInf;
      lv[u] = ok ? a.part_l[pr] : 0.f;
      ov[u] = ok ? *reinterpret_cast<const f32x4*>(a.part_o + pr * D + d) : f32x4{0.f, 0.f, 0.f, 0.f};
    }
    // running merge: rescale what is accumulated to the new maximum
    float Mb = M;
#pragma unroll
    for (int u = 0; u < kBatch; ++u) Mb = fmaxf(Mb, mv[u]);
    const float keep = M == kNegInf ? 0.f : __builtin_amdgcn_exp2f(M - Mb);
    acc *= keep;
    Ls *= keep;
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const float e = mv[u] == kNegInf ? 0.f : __builtin_amdgcn_exp2f(mv[u] - Mb);
      acc += ov[u] * e;
      Ls += lv[u] * e;
    }
    M = Mb;
  }
  const float inv = 1.f / Ls;
  acc *= inv;
  if (a.attn_out) *reinterpret_cast<f32x4*>(a.attn_out + gi) = acc;
#pragma unroll
  for (int i = 0; i < 4; ++i) Elem<T>::store_sum(a.x_out, gi + i, hv[i], acc[i]);
  if (a.x_copy) {
#pragma unroll
    for (int i = 0; i < 4; ++i) Elem<T>::store_sum(a.x_copy, gi + i, hv[i], acc[i]);
  }
}

template <typename T, int D>
static hipError_t launch_nb(int nb, dim3 grid, int threads, size_t lds, const AttnArgs& a, hipStream_t s,
                            hipEvent_t ev_start) {
  const bool flat = a.flat > 0;
  switch (nb) {
    case 1:
      return flat ? launch_k(tree_attn_kernel<T, D, 1, true>, grid, dim3(threads), lds, s, ev_start, nullptr, a)
                  : launch_k(tree_attn_kernel<T, D, 1, false>, grid, dim3(threads), lds, s, ev_start, nullptr, a);
    case 2:
      return flat ? launch_k(tree_attn_kernel<T, D, 2, true>, grid, dim3(threads), lds, s, ev_start, nullptr, a)
                  : launch_k(tree_attn_kernel<T, D, 2, false>, grid, dim3(threads), lds, s, ev_start, nullptr, a);
    default: return hipErrorInvalidValue;
  }
}

template <typename T, int D>
static hipError_t set_lds_nb(int nb, size_t lds) {
  const void* f[2] = {nullptr, nullptr};
  switch (nb) {
    case 1:
      f[0] = reinterpret_cast<const void*>(&tree_attn_kernel<T, D, 1, false>);
      f[1] = reinterpret_cast<const void*>(&tree_attn_kernel<T, D, 1, true>);
      break;
    case 2:
      f[0] = reinterpret_cast<const void*>(&tree_attn_kernel<T, D, 2, false>);
      f[1] = reinterpret_cast<const void*>(&tree_attn_kernel<T, D, 2, true>);
      break;
    default: return hipErrorInvalidValue;
  }
  for (const void* k : f) {
    const hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_tree_attn(int dtype, int head_dim, int nb, dim3 grid, int threads, size_t lds,
                            const AttnArgs& a, hipStream_t s, hipEvent_t ev_start) {
  if (dtype == 1 && head_dim == 128) return launch_nb<bf16_t, 128>(nb, grid, threads, lds, a, s, ev_start);
  if (dtype == 1 && head_dim == 64) return launch_nb<bf16_t, 64>(nb, grid, threads, lds, a, s, ev_start);
  if (dtype == 0 && head_dim == 128) return launch_nb<float, 128>(nb, grid, threads, lds, a, s, ev_start);
  if (dtype == 0 && head_dim == 64) return launch_nb<float, 64>(nb, grid, threads, lds, a, s, ev_start);
  return hipErrorInvalidValue;
}

// Ring forms (slots, key groups, tiles per group and pass): one key group takes
// three tiles per pass, two key groups two tiles each, from ten slots.
template <int D>
static hipError_t shared_ring(int stages, int kg, bool launch, dim3 grid, int threads, size_t lds, const AttnArgs& a,
                              hipStream_t s, hipEvent_t ev_start) {
  const void* f = nullptr;
  if (stages == kSharedStages1 && kg == 1)
    f = reinterpret_cast<const void*>(&tree_attn_shared_kernel<D, 2, kSharedStages1, 1, 3>);
  if (stages == kSharedStages2 && kg == 2)
    f = reinterpret_cast<const void*>(&tree_attn_shared_kernel<D, 2, kSharedStages2, 2, 2>);
  if (!f) return hipErrorInvalidValue;
  if (!launch) return hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (kg == 1)
    return launch_k(tree_attn_shared_kernel<D, 2, kSharedStages1, 1, 3>, grid, dim3(threads), lds, s, ev_start,
                    nullptr, a);
  return launch_k(tree_attn_shared_kernel<D, 2, kSharedStages2, 2, 2>, grid, dim3(threads), lds, s, ev_start, nullptr,
                  a);
}

hipError_t launch_tree_attn_shared(int head_dim, int nb, int stages, int kg, dim3 grid, int threads, size_t lds,
                                   const AttnArgs& a, hipStream_t s, hipEvent_t ev_start) {
  if (nb != 2 || threads < 128 || threads > 512 || threads % 64 || threads != 64 * a.wr * kg)
    return hipErrorInvalidValue;  // 2..8 waves
  if (lds < (size_t)shared_ring_bytes(head_dim, stages)) return hipErrorInvalidValue;
  if (head_dim == 128) return shared_ring<128>(stages, kg, true, grid, threads, lds, a, s, ev_start);
  if (head_dim == 64) return shared_ring<64>(stages, kg, true, grid, threads, lds, a, s, ev_start);
  return hipErrorInvalidValue;
}

hipError_t set_tree_attn_shared_lds_limit(int head_dim, int stages, int kg, size_t lds) {
  const AttnArgs none{};
  if (head_dim == 128) return shared_ring<128>(stages, kg, false, dim3(), 0, lds, none, nullptr, nullptr);
  if (head_dim == 64) return shared_ring<64>(stages, kg, false, dim3(), 0, lds, none, nullptr, nullptr);
  return hipErrorInvalidValue;
}

hipError_t launch_attn_merge(int dtype, int head_dim, dim3 grid, const AttnArgs& a, hipStream_t s,
                             hipEvent_t ev_stop) {
  const dim3 blk(256);
  if (dtype == 1 && head_dim == 128) return launch_k(attn_merge_kernel<bf16_t, 128>, grid, blk, 0, s, nullptr, ev_stop, a);
  if (dtype == 1 && head_dim == 64) return launch_k(attn_merge_kernel<bf16_t, 64>, grid, blk, 0, s, nullptr, ev_stop, a);
  if (dtype == 0 && head_dim == 128) return launch_k(attn_merge_kernel<float, 128>, grid, blk, 0, s, nullptr, ev_stop, a);
  if (dtype == 0 && head_dim == 64) return launch_k(attn_merge_kernel<float, 64>, grid, blk, 0, s, nullptr, ev_stop, a);
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
