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
//     unnormalised partial (O, max, sum); the last workgroup of a (b, g, row
//     block) to finish (device-scope ticket) merges all splits, writes O and
//     x, and resets the ticket to zero for the next step.
#include "common.hpp"
#include "kernels.hpp"

namespace respec {

template <typename T, int D, int NB>
__global__ __launch_bounds__(256) void tree_attn_kernel(AttnArgs a) {
  constexpr int ES = Elem<T>::kBytes;
  constexpr int E16 = 16 / ES;         // elements per 16-byte piece
  constexpr int KCH = D * ES / 64;     // 64-byte K-chunks per head row
  constexpr int DB = D / 16;           // 16-wide output blocks along D
  constexpr int CPR = D * ES / 16;     // 16-byte pieces per KV row
  constexpr int VPL = CPR / 8;         // (piece, 4-row quad) pairs per lane per tile
  constexpr int VTS = kKvTile + kVtPad;  // elements per transposed-V row
  constexpr int RB = 16 * NB;          // query rows per wave
  static_assert(VPL >= 1, "head_dim too small");

  extern __shared__ __align__(16) unsigned char smem[];
  uint32_t* s_anc = reinterpret_cast<uint32_t*>(smem);           // [kMaxNodes][4]
  int* s_ticket = reinterpret_cast<int*>(smem + kMaxNodes * 16); // [1]
  unsigned char* s_work = smem + kMaxNodes * 16 + 64;

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

  // Ancestor-or-self bitsets of the sequence's nodes (parent walk, bounded).
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
      const int p = a.parent[node0 + x];
      if (p < 0 || p >= x) break;
      x = p;
    }
    s_anc[t * 4 + 0] = w0;
    s_anc[t * 4 + 1] = w1;
    s_anc[t * 4 + 2] = w2;
    s_anc[t * 4 + 3] = w3;
  }
  __syncthreads();

  // Query fragments: lane row r = row_wave + 16*nb + lr.
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

  const size_t head_row0 = ((size_t)b * a.n_kv_heads + g) * (size_t)a.kv_cap;
  const char* kbase = reinterpret_cast<const char*>(a.k_cache) + head_row0 * D * ES;
  const char* vbase = reinterpret_cast<const char*>(a.v_cache) + head_row0 * D * ES;
  const int t_rows = L + n_nodes;
  const int kv_lo = split * a.chunk;
  const int kv_hi = min(kv_lo + a.chunk, t_rows);

  T* vt = reinterpret_cast<T*>(s_work + (size_t)wave * D * VTS * ES);

  float m_run[NB], l_run[NB];
  f32x4 o[DB][NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    m_run[nb] = kNegInf;
    l_run[nb] = 0.f;
#pragma unroll
    for (int db = 0; db < DB; ++db) o[db][nb] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  for (int t0 = kv_lo + wk * kKvTile; t0 < kv_hi; t0 += kKvTile * a.wk) {
    // K fragments: rows t0 + 16*kb + lr
    u32x4 kf[2][KCH];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const int p = t0 + 16 * kb + lr;
      if (p < kv_hi) {
        const char* src = kbase + (size_t)p * D * ES;
#pragma unroll
        for (int kc = 0; kc < KCH; ++kc) kf[kb][kc] = ld16(src + kc * 64 + lg * 16);
      } else {
#pragma unroll
        for (int kc = 0; kc < KCH; ++kc) kf[kb][kc] = u32x4{0, 0, 0, 0};
      }
    }
    // V rows for the transpose: lane holds piece c of rows 4*qd .. 4*qd+3
    u32x4 vr[VPL][4];
#pragma unroll
    for (int t = 0; t < VPL; ++t) {
      const int pair = lane + 64 * t;
      const int c = pair % CPR, qd = pair / CPR;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int p = t0 + 4 * qd + r;
        vr[t][r] = p < kv_hi ? ld16(vbase + (size_t)p * D * ES + c * 16) : u32x4{0, 0, 0, 0};
      }
    }
    // write V^T: vt[d][kv]
#pragma unroll
    for (int t = 0; t < VPL; ++t) {
      const int pair = lane + 64 * t;
      const int c = pair % CPR, qd = pair / CPR;
#pragma unroll
      for (int e = 0; e < E16; ++e) {
        const int d = c * E16 + e;
        if constexpr (ES == 2) {
          const int w = e >> 1, sh = (e & 1) * 16;
          const uint32_t h0 = (vr[t][0][w] >> sh) & 0xFFFFu, h1 = (vr[t][1][w] >> sh) & 0xFFFFu;
          const uint32_t h2 = (vr[t][2][w] >> sh) & 0xFFFFu, h3 = (vr[t][3][w] >> sh) & 0xFFFFu;
          *reinterpret_cast<u32x2*>(vt + d * VTS + 4 * qd) = u32x2{h0 | (h1 << 16), h2 | (h3 << 16)};
        } else {
          *reinterpret_cast<u32x4*>(vt + d * VTS + 4 * qd) =
              u32x4{vr[t][0][e], vr[t][1][e], vr[t][2][e], vr[t][3][e]};
        }
      }
    }
    wave_lds_sync();

    // S^T = K Q^T: lane holds S[query 16*nb + lr][kv t0 + 16*kb + 4*lg + i]
    f32x4 s[2][NB];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kc = 0; kc < KCH; ++kc) acc = mma_k64(T{}, kf[kb][kc], qf[nb][kc], acc);
        s[kb][nb] = acc;
      }
    }
    // scale + tree mask
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int p = t0 + 16 * kb + 4 * lg + i;
        const bool in = p < kv_hi;
        const int ai = p - L;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          bool vis = in;
          if (in && ai >= 0) {
            vis = qnode[nb] >= 0 && ((s_anc[qnode[nb] * 4 + (ai >> 5)] >> (ai & 31)) & 1u);
          }
          s[kb][nb][i] = vis ? s[kb][nb][i] * a.scale_log2 : kNegInf;
        }
      }
    }
    // online softmax (row max shared by the 4 lane groups of a row)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      float tm = kNegInf;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) tm = fmaxf(tm, s[kb][nb][i]);
      tm = fmaxf(tm, __shfl_xor(tm, 16, 64));
      tm = fmaxf(tm, __shfl_xor(tm, 32, 64));
      const float mn = fmaxf(m_run[nb], tm);
      const bool none = mn == kNegInf;
      const float alpha = none ? 1.f : __builtin_amdgcn_exp2f(m_run[nb] - mn);
      float ps = 0.f;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float pv = none ? 0.f : __builtin_amdgcn_exp2f(s[kb][nb][i] - mn);
          s[kb][nb][i] = pv;
          ps += pv;
        }
      l_run[nb] = l_run[nb] * alpha + ps;
      m_run[nb] = mn;
#pragma unroll
      for (int db = 0; db < DB; ++db) o[db][nb] *= alpha;
    }

    // O^T += V^T P^T: k order per lane = kv {4lg+i (kb 0), 16+4lg+i (kb 1)}
    if constexpr (ES == 2) {
      u32x4 phi[NB], plo[NB];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        uint32_t hi16[8], lo16[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float pv = s[j >> 2][nb][j & 3];
          const uint16_t hb = f32_to_bf16(pv);
          hi16[j] = hb;
          lo16[j] = f32_to_bf16(pv - bf16_to_f32(hb));
        }
        phi[nb] = u32x4{hi16[0] | (hi16[1] << 16), hi16[2] | (hi16[3] << 16), hi16[4] | (hi16[5] << 16),
                        hi16[6] | (hi16[7] << 16)};
        plo[nb] = u32x4{lo16[0] | (lo16[1] << 16), lo16[2] | (lo16[3] << 16), lo16[4] | (lo16[5] << 16),
                        lo16[6] | (lo16[7] << 16)};
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
      for (int db = 0; db < DB; ++db)
        *reinterpret_cast<f32x4*>(a.part_o + (pbase + rl) * D + 16 * db + 4 * lg) = o[db][nb];
      if (lg == 0) {
        a.part_m[pbase + rl] = m_run[nb];
        a.part_l[pbase + rl] = l_run[nb];
      }
    }
  } else {
    __syncthreads();  // every wave is done with its V^T tile
    float* mo = reinterpret_cast<float*>(s_work);  // [nwaves][RB][D]
    float* mm = mo + (size_t)nwaves * RB * D;     // [nwaves][RB]
    float* ml = mm + nwaves * RB;
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
    for (int idx = threadIdx.x; idx < a.rows_per_wg * D; idx += blockDim.x) {
      const int rl = idx / D, d = idx - rl * D;
      const int gr = rl / RB, rr = rl - gr * RB;
      float M = kNegInf;
      for (int k = 0; k < a.wk; ++k) M = fmaxf(M, mm[(gr + a.wr * k) * RB + rr]);
      float Os = 0.f, Ls = 0.f;
      if (M != kNegInf) {
        for (int k = 0; k < a.wk; ++k) {
          const int wv = gr + a.wr * k;
          const float sc = __builtin_amdgcn_exp2f(mm[wv * RB + rr] - M);
          Os += mo[((size_t)wv * RB + rr) * D + d] * sc;
          Ls += ml[wv * RB + rr] * sc;
        }
      }
      a.part_o[(pbase + rl) * D + d] = Os;
      if (d == 0) {
        a.part_m[pbase + rl] = M;
        a.part_l[pbase + rl] = Ls;
      }
    }
  }

  // ---- completion ticket; the last split merges ----
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) *s_ticket = atomicAdd(a.counter + bgr, 1);
  __syncthreads();
  if (*s_ticket != a.nsplit - 1) return;
  __threadfence();

  const int rows_here = min(a.rows_per_wg, R - row_wg);
  const size_t sbase = (size_t)bgr * a.nsplit * a.rows_per_wg;
  for (int idx = threadIdx.x; idx < rows_here * D; idx += blockDim.x) {
    const int rl = idx / D, d = idx - rl * D;
    float M = kNegInf;
    for (int s = 0; s < a.nsplit; ++s) M = fmaxf(M, a.part_m[sbase + (size_t)s * a.rows_per_wg + rl]);
    float Os = 0.f, Ls = 0.f;
    for (int s = 0; s < a.nsplit; ++s) {
      const size_t pr = sbase + (size_t)s * a.rows_per_wg + rl;
      const float sc = __builtin_amdgcn_exp2f(a.part_m[pr] - M);
      Ls += a.part_l[pr] * sc;
      Os += a.part_o[pr * D + d] * sc;
    }
    const float O = Os / Ls;
    const int r = row_wg + rl;
    const int node = r / a.group;
    const int h = g * a.group + (r - node * a.group);
    const size_t gi = (size_t)(node0 + node) * a.hidden_size + (size_t)h * D + d;
    if (a.attn_out) a.attn_out[gi] = O;
    const float hv = Elem<T>::to_f32(a.hidden, gi);
    Elem<T>::store(a.x_out, gi, hv + O);
  }
  if (threadIdx.x == 0) a.counter[bgr] = 0;
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
