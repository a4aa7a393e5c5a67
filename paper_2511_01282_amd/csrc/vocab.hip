// Fused vocabulary pass and path reduction of a draft-tree verification step.
//
// Per node row i (ReSpec: entropy of Eq. 1; relaxed check of Eq. 6-7;
// look-ahead tolerance of Section 3.4; winner of Algorithm 1's RelaxedVerify):
//   1. chunk workgroups stream z[i][chunk] once: online max m, argmax (smallest
//      id on ties), S = sum e^(z-m), T = sum e^(z-m)(z-m), and a top-KO list;
//   2. the last chunk workgroup of the row (device-scope ticket) merges the
//      partials: lse = m + log S, entropy = log S - T/S, top-k by (z desc, id
//      asc); then, for every child j of node i, the predicates of j's token:
//      GREEDY (t == argmax), TOPK (t among the first k), TAU (z_max - z_t <= tau,
//      compared in double), RELAXED (retrieved and TOPK and TAU);
//   3. the last row of a sequence runs the look-ahead procedure on every
//      root-to-leaf chain (64-bit chain masks, one lane per leaf) and picks the
//      winner: longest accepted length, then smallest last accepted node, then
//      smallest leaf.
// Extra workgroups (one per sequence) report sequences whose node range is
// unusable, since no row workgroup would finish them.
#include "common.hpp"
#include "kernels.hpp"

namespace respec {

namespace {

constexpr int kFlagGreedy = 1, kFlagTopk = 2, kFlagTau = 4, kFlagRelaxed = 8, kFlagOnPath = 16;
constexpr int kStatusTree = 5, kStatusCapacity = 6, kStatusToken = 9;

__device__ __forceinline__ void merge_stats(float& m, float& S, float& T, int& am, float m2, float S2, float T2,
                                            int am2) {
  if (m2 == kNegInf) return;
  if (m == kNegInf) {
    m = m2; S = S2; T = T2; am = am2;
    return;
  }
  const float M = fmaxf(m, m2);
  const float d1 = m - M, d2 = m2 - M;
  const float e1 = __expf(d1), e2 = __expf(d2);
  T = e1 * (T + d1 * S) + e2 * (T2 + d2 * S2);
  S = e1 * S + e2 * S2;
  am = (m > m2) ? am : (m2 > m) ? am2 : min(am, am2);
  m = M;
}

__device__ __forceinline__ void wave_merge_stats(float& m, float& S, float& T, int& am) {
  for (int off = 32; off > 0; off >>= 1) {
    const float m2 = __shfl_xor(m, off, 64), S2 = __shfl_xor(S, off, 64), T2 = __shfl_xor(T, off, 64);
    const int am2 = __shfl_xor(am, off, 64);
    merge_stats(m, S, T, am, m2, S2, T2, am2);
  }
}

__device__ __forceinline__ void wave_best(float& v, int& id) {
  for (int off = 32; off > 0; off >>= 1) {
    const float ov = __shfl_xor(v, off, 64);
    const int oi = __shfl_xor(id, off, 64);
    if (better(ov, oi, v, id)) {
      v = ov;
      id = oi;
    }
  }
}

// K rounds of wave-wide selection over per-lane sorted lists (tv, ti).
template <int KO>
__device__ __forceinline__ void wave_topk(float (&tv)[KO], int (&ti)[KO], float (&rv)[KO], int (&ri)[KO]) {
#pragma unroll
  for (int k = 0; k < KO; ++k) {
    float bv = tv[0];
    int bi = ti[0];
    wave_best(bv, bi);
    rv[k] = bv;
    ri[k] = bi;
    const bool own = bv != kNegInf && ti[0] == bi;
#pragma unroll
    for (int q = 0; q < KO - 1; ++q) {
      tv[q] = own ? tv[q + 1] : tv[q];
      ti[q] = own ? ti[q + 1] : ti[q];
    }
    tv[KO - 1] = own ? kNegInf : tv[KO - 1];
    ti[KO - 1] = own ? INT_MAX : ti[KO - 1];
  }
}

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t x) {
  for (int off = 32; off > 0; off >>= 1) {
    const uint32_t lo = __shfl_xor((uint32_t)x, off, 64), hi = __shfl_xor((uint32_t)(x >> 32), off, 64);
    const uint64_t y = ((uint64_t)hi << 32) | lo;
    x = y < x ? y : x;
  }
  return x;
}

// Look-ahead tolerance on one chain u_1..u_d; bit s-1 of G / OK describes u_s.
__device__ __forceinline__ int lookahead_bits(int d, uint64_t G, uint64_t OK, int m, int phi) {
  int l0 = 0;
  while (l0 < d && ((G >> l0) & 1ull)) ++l0;
  int cur = l0, last = l0;
  for (int att = 0; att < phi && cur < d; ++att) {
    if (!((OK >> cur) & 1ull)) break;
    int xi = 0;
    while (cur + 1 + xi < d && ((G >> (cur + 1 + xi)) & 1ull)) ++xi;
    if (xi >= m) {
      last = cur + 1 + xi;
      cur = last;
    } else {
      cur = cur + 1;
    }
  }
  return last;
}

// node_off describes B disjoint, consecutive, non-empty node ranges covering [0, M)
__device__ __forceinline__ bool layout_ok(const VocabArgs& a) {
  if (a.node_off[0] != 0 || a.node_off[a.batch] != a.total_nodes) return false;
  for (int b = 0; b < a.batch; ++b) {
    const int n = a.node_off[b + 1] - a.node_off[b];
    if (n < 1 || n > a.max_nodes) return false;
  }
  return true;
}

__device__ void write_seq_error(const VocabArgs& a, int b, int status, int n0, int n, int lane) {
  for (int s = lane; s <= a.max_depth; s += 64) a.path[(size_t)b * (a.max_depth + 1) + s] = -1;
  for (int j = lane; j < n; j += 64) {
    a.leaf_acc_len[n0 + j] = -1;
    a.flags[n0 + j] = 0;
  }
  if (lane == 0) {
    a.acc_len[b] = -1;
    a.bonus[b] = -1;
    a.winner_leaf[b] = -1;
    a.seq_status[b] = status;
  }
}

// One wave: validate sequence b and reduce its accepted path.
__device__ void path_reduce(const VocabArgs& a, int b, int n0, int n, uint8_t* s_hc, int lane) {
  bool bad_tree = false, bad_tok = false;
  for (int j = lane; j < n; j += 64) {
    const int p = a.parent[n0 + j];
    if (j == 0) {
      bad_tree |= p != -1;
    } else {
      bad_tree |= p < 0 || p >= j;
      const int t = a.token[n0 + j];
      bad_tok |= t < 0 || t >= a.vocab || a.src[n0 + j] > 1;
    }
  }
  bad_tree = __any(bad_tree);
  if (!bad_tree) {
    for (int j = lane; j < n; j += 64) {
      int d = 0, x = j;
      while (x != 0) {
        x = a.parent[n0 + x];
        ++d;
      }
      bad_tree |= d > a.max_depth;
    }
    bad_tree = __any(bad_tree);
  }
  bad_tok = __any(bad_tok);
  const int L = a.kv_len[b];
  const bool bad_cap = L < 0 || L > a.max_kv || L > a.kv_cap - n;
  const int status = bad_tree ? kStatusTree : bad_tok ? kStatusToken : bad_cap ? kStatusCapacity : 0;
  if (status != 0) {
    write_seq_error(a, b, status, n0, n, lane);
    return;
  }

  for (int j = lane; j < n; j += 64) s_hc[j] = 0;
  wave_lds_sync();
  for (int j = lane; j < n; j += 64)
    if (j > 0) s_hc[a.parent[n0 + j]] = 1;
  wave_lds_sync();

  uint64_t best = ~0ull;
  for (int j = lane; j < n; j += 64) {
    if (s_hc[j]) {
      a.leaf_acc_len[n0 + j] = -1;
      continue;
    }
    int d = 0;
    for (int x = j; x != 0; x = a.parent[n0 + x]) ++d;
    uint64_t G = 0, OK = 0;
    int s = d;
    for (int x = j; x != 0; x = a.parent[n0 + x], --s) {
      const uint32_t f = a.flags[n0 + x];
      G |= (uint64_t)(f & kFlagGreedy) << (s - 1);
      OK |= (uint64_t)((f & (kFlagGreedy | kFlagRelaxed)) != 0) << (s - 1);
    }
    const int acc = lookahead_bits(d, G, OK, a.min_lookahead, a.max_relaxed);
    int e = j;
    for (int q = 0; q < d - acc; ++q) e = a.parent[n0 + e];
    a.leaf_acc_len[n0 + j] = acc;
    const uint64_t key = ((uint64_t)(kMaxDepth - acc) << 40) | ((uint64_t)e << 20) | (uint64_t)j;
    best = key < best ? key : best;
  }
  best = wave_min_u64(best);
  const int acc = kMaxDepth - (int)(best >> 40);
  const int e = (int)((best >> 20) & 0xFFFFFull);
  const int leaf = (int)(best & 0xFFFFFull);
  for (int s = acc + 1 + lane; s <= a.max_depth; s += 64) a.path[(size_t)b * (a.max_depth + 1) + s] = -1;
  if (lane == 0) {
    int x = e;
    for (int s = acc; s >= 0; --s) {
      a.path[(size_t)b * (a.max_depth + 1) + s] = x;
      a.flags[n0 + x] = (uint8_t)(a.flags[n0 + x] | kFlagOnPath);
      x = s > 0 ? a.parent[n0 + x] : x;
    }
    a.acc_len[b] = acc;
    a.bonus[b] = a.argmax[n0 + e];
    a.winner_leaf[b] = leaf;
    a.seq_status[b] = 0;
  }
}

}  // namespace

template <int KO>
__global__ __launch_bounds__(256) void vocab_kernel(VocabArgs a) {
  __shared__ float s_st[4][4];
  __shared__ int s_am[4];
  __shared__ float s_tv[4 * KO];
  __shared__ int s_ti[4 * KO];
  __shared__ int s_ticket;
  __shared__ uint8_t s_hc[kMaxNodes];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nwaves = blockDim.x >> 6;
  const bool lay_ok = layout_ok(a);

  if (blockIdx.y >= (unsigned)a.total_nodes) {
    // sequence report: only sequences that no row workgroup can finish
    const int b = blockIdx.y - a.total_nodes;
    if (blockIdx.x != 0 || wave != 0 || b >= a.batch || lay_ok) return;
    write_seq_error(a, b, kStatusTree, 0, 0, lane);
    return;
  }

  const int i = blockIdx.y, c = blockIdx.x;
  const float* z = a.logits + (size_t)i * a.vocab;
  const int lo = c * a.chunk, hi = min(a.vocab, lo + a.chunk);

  float m = kNegInf, S = 0.f, T = 0.f;
  int am = INT_MAX;
  float tv[KO];
  int ti[KO];
#pragma unroll
  for (int k = 0; k < KO; ++k) {
    tv[k] = kNegInf;
    ti[k] = INT_MAX;
  }
  for (int v = lo + threadIdx.x; v < hi; v += blockDim.x) {
    const float x = z[v];
    if (x > m) {
      if (m == kNegInf) {
        S = 1.f;
        T = 0.f;
      } else {
        const float d = m - x;
        const float sc = __expf(d);
        T = sc * (T + d * S);
        S = sc * S + 1.f;
      }
      m = x;
      am = v;
    } else {
      const float d = x - m;
      const float e = __expf(d);
      S += e;
      T += e * d;
    }
    if (x > tv[KO - 1]) {
      tv[KO - 1] = x;
      ti[KO - 1] = v;
#pragma unroll
      for (int k = KO - 1; k > 0; --k) {
        const bool sw = tv[k] > tv[k - 1];
        const float a0 = tv[k - 1], a1 = tv[k];
        const int b0 = ti[k - 1], b1 = ti[k];
        tv[k - 1] = sw ? a1 : a0;
        tv[k] = sw ? a0 : a1;
        ti[k - 1] = sw ? b1 : b0;
        ti[k] = sw ? b0 : b1;
      }
    }
  }
  wave_merge_stats(m, S, T, am);
  float rv[KO];
  int ri[KO];
  wave_topk<KO>(tv, ti, rv, ri);
  if (lane == 0) {
    s_st[wave][0] = m;
    s_st[wave][1] = S;
    s_st[wave][2] = T;
    s_am[wave] = am;
  }
#pragma unroll
  for (int k = 0; k < KO; ++k)
    if (lane == k) {
      s_tv[wave * KO + k] = rv[k];
      s_ti[wave * KO + k] = ri[k];
    }
  __syncthreads();

  const size_t pidx = (size_t)i * a.nchunk + c;
  if (wave == 0) {
    if (lane < nwaves) {
      m = s_st[lane][0];
      S = s_st[lane][1];
      T = s_st[lane][2];
      am = s_am[lane];
    } else {
      m = kNegInf;
      S = 0.f;
      T = 0.f;
      am = INT_MAX;
    }
    wave_merge_stats(m, S, T, am);
    // one candidate per lane, KO rounds
    float cv[1];
    int ci[1];
    cv[0] = lane < nwaves * KO ? s_tv[lane] : kNegInf;
    ci[0] = lane < nwaves * KO ? s_ti[lane] : INT_MAX;
#pragma unroll
    for (int k = 0; k < KO; ++k) {
      float bv = cv[0];
      int bi = ci[0];
      wave_best(bv, bi);
      rv[k] = bv;
      ri[k] = bi;
      if (bv != kNegInf && ci[0] == bi) {
        cv[0] = kNegInf;
        ci[0] = INT_MAX;
      }
    }
    if (lane == 0) {
      a.p_m[pidx] = m;
      a.p_s[pidx] = S;
      a.p_t[pidx] = T;
      a.p_am[pidx] = am;
    }
#pragma unroll
    for (int k = 0; k < KO; ++k)
      if (lane == k) {
        a.p_tv[pidx * KO + k] = rv[k];
        a.p_ti[pidx * KO + k] = ri[k];
      }
  }

  // ---- row completion ticket ----
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) s_ticket = atomicAdd(a.row_counter + i, 1);
  __syncthreads();
  if (s_ticket != a.nchunk - 1 || wave != 0) return;
  __threadfence();

  if (lane < a.nchunk) {
    const size_t q = (size_t)i * a.nchunk + lane;
    m = a.p_m[q];
    S = a.p_s[q];
    T = a.p_t[q];
    am = a.p_am[q];
#pragma unroll
    for (int k = 0; k < KO; ++k) {
      tv[k] = a.p_tv[q * KO + k];
      ti[k] = a.p_ti[q * KO + k];
    }
  } else {
    m = kNegInf;
    S = 0.f;
    T = 0.f;
    am = INT_MAX;
#pragma unroll
    for (int k = 0; k < KO; ++k) {
      tv[k] = kNegInf;
      ti[k] = INT_MAX;
    }
  }
  wave_merge_stats(m, S, T, am);
  wave_topk<KO>(tv, ti, rv, ri);
  const float logS = __logf(S);
  const float lse = m + logS;
  if (lane == 0) {
    a.max_logit[i] = m;
    a.argmax[i] = am;
    a.lse[i] = lse;
    a.entropy[i] = logS - T / S;
    a.row_counter[i] = 0;
  }
#pragma unroll
  for (int k = 0; k < KO; ++k)
    if (lane == k && k < a.topk_out) {
      a.topk_id[(size_t)i * a.topk_out + k] = ri[k];
      a.topk_logprob[(size_t)i * a.topk_out + k] = rv[k] - lse;
    }
  if (!lay_ok) return;

  // sequence of row i
  int b = 0;
  while (b + 1 < a.batch && a.node_off[b + 1] <= i) ++b;
  const int n0 = a.node_off[b], n = a.node_off[b + 1] - n0;
  const int li = i - n0;

  // predicates of the children of node li
  for (int j = lane; j < n; j += 64) {
    if (j == 0) continue;
    if (a.parent[n0 + j] != li) continue;
    const int t = a.token[n0 + j];
    uint32_t f = 0;
    float lp = 0.f;
    if (t >= 0 && t < a.vocab) {
      const float zt = z[t];
      bool intop = false;
#pragma unroll
      for (int k = 0; k < KO; ++k) intop |= (k < a.topk) && (ri[k] == t);
      if (t == am) f |= kFlagGreedy;
      if (intop) f |= kFlagTopk;
      if ((double)m - (double)zt <= (double)a.tau) f |= kFlagTau;
      if (a.src[n0 + j] == 1 && (f & kFlagTopk) && (f & kFlagTau)) f |= kFlagRelaxed;
      lp = zt - lse;
    }
    a.flags[n0 + j] = (uint8_t)f;
    a.tok_logprob[n0 + j] = lp;
  }
  if (li == 0 && lane == 0) {
    a.flags[n0] = 0;
    a.tok_logprob[n0] = 0.f;
  }

  // ---- sequence completion ticket ----
  __threadfence();
  int ticket = 0;
  if (lane == 0) ticket = atomicAdd(a.seq_counter + b, 1);
  ticket = __shfl(ticket, 0, 64);
  if (ticket != n - 1) return;
  __threadfence();
  path_reduce(a, b, n0, n, s_hc, lane);
  if (lane == 0) a.seq_counter[b] = 0;
}

hipError_t launch_vocab(int ko, dim3 grid, const VocabArgs& a, hipStream_t s) {
  if (ko == 8)
    hipLaunchKernelGGL((vocab_kernel<8>), grid, dim3(256), 0, s, a);
  else if (ko == 16)
    hipLaunchKernelGGL((vocab_kernel<16>), grid, dim3(256), 0, s, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

__global__ void zero_i32_kernel(int32_t* p, size_t n) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) p[i] = 0;
}

hipError_t launch_zero_i32(int32_t* p, size_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const unsigned blocks = (unsigned)((n + 255) / 256 < 1024 ? (n + 255) / 256 : 1024);
  hipLaunchKernelGGL(zero_i32_kernel, dim3(blocks), dim3(256), 0, s, p, n);
  return hipGetLastError();
}

}  // namespace respec
