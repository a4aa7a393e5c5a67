// Row finalisation and path reduction of a draft-tree verification step.
//
// Per node row i (ReSpec: entropy of Eq. 1; relaxed check of Eq. 6-7;
// look-ahead tolerance of Section 3.4; winner of Algorithm 1's RelaxedVerify):
//   1. one workgroup merges the row's per-tile partials written by the LM-head
//      epilogue (online max / sum / entropy terms and exact top-K lists) with
//      bitonic list merges: lse = m + log S, entropy = log S - T/S, top-k by
//      (z desc, id asc); then, for every child j of node i, the predicates of
//      j's token: GREEDY (t == argmax), TOPK (t among the first k), TAU
//      (z_max - z_t <= tau, compared in double), RELAXED (retrieved and TOPK and
//      TAU);
//   2. the last row of a sequence to finish (device-scope ticket; predicates
//      handed over with device-coherent stores and loads) runs the look-ahead
//      procedure on every root-to-leaf chain (64-bit chain masks, one lane per
//      leaf) and picks the winner: longest accepted length, then smallest last
//      accepted node, then smallest leaf.
// Extra workgroups (one per sequence) report sequences whose node range is
// unusable, since no row workgroup would finish them.
#include "common.hpp"
#include "kernels.hpp"

namespace respec {

namespace {

constexpr int kFlagGreedy = 1, kFlagTopk = 2, kFlagTau = 4, kFlagRelaxed = 8, kFlagOnPath = 16;
constexpr int kStatusTree = 5, kStatusCapacity = 6, kStatusToken = 9;

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t x) {
  uint64_t y;
  y = xchg<0>(x); x = y < x ? y : x;
  y = xchg<1>(x); x = y < x ? y : x;
  y = xchg<2>(x); x = y < x ? y : x;
  y = xchg<3>(x); x = y < x ? y : x;
  y = xchg<4>(x); x = y < x ? y : x;
  y = xchg<5>(x); x = y < x ? y : x;
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

// One wave: validate sequence b and reduce its accepted path.  The sequence's
// parents, predicate bits and argmaxes are staged in LDS once; every lane walks
// its leaves' chains once (recording the chain in LDS), so no chain step
// touches global memory.
__device__ void path_reduce(const VocabArgs& a, int b, int n0, int n, int* s_par, uint8_t* s_flag, uint8_t* s_hc,
                            int* s_am, uint8_t* s_chain, int lane) {
  bool bad_tree = false, bad_tok = false;
  for (int j = lane; j < n; j += 64) {
    const int p = a.parent[n0 + j];
    s_par[j] = p;
    s_flag[j] = (uint8_t)ld_dev(a.flag_ws + n0 + j);
    s_am[j] = ld_dev(a.argmax + n0 + j);
    s_hc[j] = 0;
    if (j == 0) {
      bad_tree |= p != -1;
    } else {
      bad_tree |= p < 0 || p >= j;
      const int t = a.token[n0 + j];
      bad_tok |= t < 0 || t >= a.vocab || a.src[n0 + j] > 1;
    }
  }
  bad_tree = __any(bad_tree);
  bad_tok = __any(bad_tok);
  const int L = a.kv_len[b];
  const bool bad_cap = L < 0 || L > a.max_kv || L > a.kv_cap - n;
  uint64_t best = ~0ull;
  if (!bad_tree) {
    wave_lds_sync();
    for (int j = lane; j < n; j += 64)
      if (j > 0) s_hc[s_par[j]] = 1;
    wave_lds_sync();
    // parents strictly decrease, so every walk ends at the root within n steps
    uint8_t* chain = s_chain + lane * kMaxDepth;
    bool too_deep = false;
    for (int j = lane; j < n; j += 64) {
      if (s_hc[j]) {
        a.leaf_acc_len[n0 + j] = -1;
        continue;
      }
      uint64_t g_rev = 0, ok_rev = 0;  // bit k describes the node k steps above the leaf
      int d = 0, x = j;
      while (x != 0 && d < kMaxDepth) {
        chain[d] = (uint8_t)x;
        const uint32_t f = s_flag[x];
        g_rev |= (uint64_t)(f & kFlagGreedy) << d;
        ok_rev |= (uint64_t)((f & (kFlagGreedy | kFlagRelaxed)) != 0) << d;
        x = s_par[x];
        ++d;
      }
      if (x != 0 || d > a.max_depth) {
        too_deep = true;
        continue;
      }
      // bit s-1 of G / OK describes u_s, the node at depth s
      const uint64_t G = d ? (__builtin_bitreverse64(g_rev) >> (64 - d)) : 0ull;
      const uint64_t OK = d ? (__builtin_bitreverse64(ok_rev) >> (64 - d)) : 0ull;
      const int acc = lookahead_bits(d, G, OK, a.min_lookahead, a.max_relaxed);
      const int e = acc == 0 ? 0 : chain[d - acc];
      a.leaf_acc_len[n0 + j] = acc;
      const uint64_t key = ((uint64_t)(kMaxDepth - acc) << 40) | ((uint64_t)e << 20) | (uint64_t)j;
      best = key < best ? key : best;
    }
    bad_tree = __any(too_deep);
  }
  const int status = bad_tree ? kStatusTree : bad_tok ? kStatusToken : bad_cap ? kStatusCapacity : 0;
  if (status != 0) {
    write_seq_error(a, b, status, n0, n, lane);
    return;
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
      s_flag[x] = (uint8_t)(s_flag[x] | kFlagOnPath);
      x = s > 0 ? s_par[x] : x;
    }
    a.acc_len[b] = acc;
    a.bonus[b] = s_am[e];
    a.winner_leaf[b] = leaf;
    a.seq_status[b] = 0;
  }
  wave_lds_sync();
  for (int j = lane; j < n; j += 64) a.flags[n0 + j] = s_flag[j];
}

}  // namespace

template <int KO>
__global__ __launch_bounds__(256) void finalize_kernel(VocabArgs a) {
  constexpr int W = TilePartial<KO>::kWords;
  __shared__ float s_st[4][4];
  __shared__ uint64_t s_key[4][KO];
  __shared__ int s_par[kMaxNodes];
  __shared__ int s_node_am[kMaxNodes];
  __shared__ uint8_t s_flag[kMaxNodes];
  __shared__ uint8_t s_hc[kMaxNodes];
  __shared__ uint8_t s_chain[64 * kMaxDepth];

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nwaves = blockDim.x >> 6;
  const bool lay_ok = layout_ok(a);

  if (blockIdx.x >= (unsigned)a.total_nodes) {
    // sequence report: only sequences that no row workgroup can finish
    const int b = blockIdx.x - a.total_nodes;
    if (wave != 0 || b >= a.batch || lay_ok) return;
    write_seq_error(a, b, kStatusTree, 0, 0, lane);
    return;
  }

  const int i = blockIdx.x;
  const float* z = a.logits + (size_t)i * a.vocab;

  // The row's children: prefetch (wave 0) their parents, tokens, tags and logits z[t].
  int b = 0, n0 = 0, n = 0;
  if (lay_ok) {
    while (b + 1 < a.batch && a.node_off[b + 1] <= i) ++b;
    n0 = a.node_off[b];
    n = a.node_off[b + 1] - n0;
  }
  const int li = i - n0;
  int c_par[2], c_tok[2], c_src[2];
  float c_z[2];
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int j = lane + 64 * q;
    c_par[q] = -2;
    c_tok[q] = -1;
    c_src[q] = 0;
    c_z[q] = 0.f;
    if (wave == 0 && lay_ok && j < n) {
      c_par[q] = a.parent[n0 + j];
      if (j > 0 && c_par[q] == li) {
        c_tok[q] = a.token[n0 + j];
        c_src[q] = a.src[n0 + j];
        if (c_tok[q] >= 0 && c_tok[q] < a.vocab) c_z[q] = z[c_tok[q]];
      }
    }
  }

  // merge the row's tile partials: each thread folds its tiles, then the waves
  RowStats st;
  st.init();
  uint64_t key[KO];
#pragma unroll
  for (int k = 0; k < KO; ++k) key[k] = 0ull;
  const uint32_t* prow = reinterpret_cast<const uint32_t*>(a.partials) + (size_t)i * a.n_vtiles * W;
  constexpr int kLoadBatch = 2;
  for (int t0 = threadIdx.x; t0 < a.n_vtiles; t0 += kLoadBatch * blockDim.x) {
    u32x4 buf[kLoadBatch][W / 4];
#pragma unroll
    for (int u = 0; u < kLoadBatch; ++u) {
      const int t = t0 + u * blockDim.x;
#pragma unroll
      for (int q = 0; q < W / 4; ++q)
        buf[u][q] = t < a.n_vtiles ? *reinterpret_cast<const u32x4*>(prow + (size_t)t * W + 4 * q)
                                   : u32x4{__float_as_uint(kNegInf), 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < kLoadBatch; ++u) {
      st.merge(__uint_as_float(buf[u][0][0]), __uint_as_float(buf[u][0][1]), __uint_as_float(buf[u][0][2]),
               (int)buf[u][0][3]);
      uint64_t pk[KO];
#pragma unroll
      for (int k = 0; k < KO; ++k) {
        const u32x4 w4 = buf[u][1 + k / 2];
        pk[k] = (k & 1) ? (((uint64_t)w4[3] << 32) | w4[2]) : (((uint64_t)w4[1] << 32) | w4[0]);
      }
      merge_topk<KO>(key, pk);
    }
  }
  st.merge_level<0>();
  merge_topk_level<KO, 0>(key);
  st.merge_level<1>();
  merge_topk_level<KO, 1>(key);
  st.merge_level<2>();
  merge_topk_level<KO, 2>(key);
  st.merge_level<3>();
  merge_topk_level<KO, 3>(key);
  st.merge_level<4>();
  merge_topk_level<KO, 4>(key);
  st.merge_level<5>();
  merge_topk_level<KO, 5>(key);
  if (lane == 0) {
    s_st[wave][0] = st.m;
    s_st[wave][1] = st.S;
    s_st[wave][2] = st.T;
    s_st[wave][3] = __int_as_float(st.am);
#pragma unroll
    for (int k = 0; k < KO; ++k) s_key[wave][k] = key[k];
  }
  __syncthreads();
  if (wave != 0) return;
  const int src_wave = lane & 3;
  st.m = s_st[src_wave][0];
  st.S = s_st[src_wave][1];
  st.T = s_st[src_wave][2];
  st.am = __float_as_int(s_st[src_wave][3]);
#pragma unroll
  for (int k = 0; k < KO; ++k) key[k] = s_key[src_wave][k];
  st.merge_level<0>();
  merge_topk_level<KO, 0>(key);
  st.merge_level<1>();
  merge_topk_level<KO, 1>(key);

  const float m = st.m;
  const int am = st.am;
  const float logS = __logf(st.S);
  const float lse = m + logS;
  if (lane == 0) {
    a.max_logit[i] = m;
    st_dev(a.argmax + i, am);
    a.lse[i] = lse;
    a.entropy[i] = logS - st.T / st.S;
  }
#pragma unroll
  for (int k = 0; k < KO; ++k)
    if (lane == k && k < a.topk_out) {
      a.topk_id[(size_t)i * a.topk_out + k] = key_id(key[k]);
      a.topk_logprob[(size_t)i * a.topk_out + k] = key_value(key[k]) - lse;
    }
  if (!lay_ok) return;

  // predicates of the children of node li (prefetched above)
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int j = lane + 64 * q;
    if (j == 0 || j >= n || c_par[q] != li) continue;
    const int t = c_tok[q];
    uint32_t f = 0;
    float lp = 0.f;
    if (t >= 0 && t < a.vocab) {
      const float zt = c_z[q];
      bool intop = false;
#pragma unroll
      for (int k = 0; k < KO; ++k) intop |= (k < a.topk) && (key_id(key[k]) == t);
      if (t == am) f |= kFlagGreedy;
      if (intop) f |= kFlagTopk;
      if ((double)m - (double)zt <= (double)a.tau) f |= kFlagTau;
      if (c_src[q] == 1 && (f & kFlagTopk) && (f & kFlagTau)) f |= kFlagRelaxed;
      lp = zt - lse;
    }
    st_dev(a.flag_ws + n0 + j, (int32_t)f);
    a.tok_logprob[n0 + j] = lp;
  }
  if (li == 0 && lane == 0) {
    st_dev(a.flag_ws + n0, 0);
    a.tok_logprob[n0] = 0.f;
  }

  // ---- sequence completion ticket ----
  stores_done();
  int ticket = 0;
  if (lane == 0) ticket = atomicAdd(a.seq_counter + b, 1);
  ticket = __shfl(ticket, 0, 64);
  if (ticket != n - 1) return;
  path_reduce(a, b, n0, n, s_par, s_flag, s_hc, s_node_am, s_chain, lane);
  if (lane == 0) st_dev(a.seq_counter + b, 0);
}

hipError_t launch_finalize(int ko, int blocks, const VocabArgs& a, hipStream_t s) {
  if (ko == 8)
    hipLaunchKernelGGL((finalize_kernel<8>), dim3(blocks), dim3(256), 0, s, a);
  else if (ko == 16)
    hipLaunchKernelGGL((finalize_kernel<16>), dim3(blocks), dim3(256), 0, s, a);
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
