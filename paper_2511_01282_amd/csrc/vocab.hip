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

// node_off describes B disjoint, consecutive, non-empty node ranges covering
// [0, M), each at most max_nodes long.  Checked lane-parallel: lane k holds
// node_off[k] and node_off[k+1] (v0, vn0: the caller's loads for k < 64, with
// k clamped to B); further groups of 64 are loaded here.  Also finds the
// sequence b of node row `row` and its range [n0, n0 + n).  Every lane of the
// wave takes part.
struct SeqLayout {
  bool ok;
  int b, n0, n;
};

__device__ __forceinline__ void load_offsets(const VocabArgs& a, int lane, int& v0, int& vn0) {
  const int k = min(lane, a.batch);
  v0 = a.node_off[k];
  vn0 = a.node_off[min(k + 1, a.batch)];
}

template <bool Wide>
__device__ __forceinline__ SeqLayout scan_layout(const VocabArgs& a, int row, int lane, int v0, int vn0) {
  SeqLayout r{true, 0, 0, 0};
  bool bad = false;
  int before = 0;  // sequences k >= 1 that start at or before row
  for (int k0 = 0; k0 <= (Wide ? a.batch : 0); k0 += 64) {
    const int k = k0 + lane;
    int v = v0, vn = vn0;
    if (Wide && k0 > 0) {
      const int kc = min(k, a.batch);
      v = a.node_off[kc];
      vn = a.node_off[min(kc + 1, a.batch)];
    }
    if (k <= a.batch) {
      if (k == 0 && v != 0) bad = true;
      if (k == a.batch && v != a.total_nodes) bad = true;
      if (k < a.batch && (vn - v < 1 || vn - v > a.max_nodes)) bad = true;
    }
    before += __popcll(__ballot(k >= 1 && k < a.batch && v <= row));
  }
  r.ok = !__any(bad);
  r.b = r.ok ? before : 0;
  if (!Wide) {
    r.n0 = __shfl(v0, r.b, 64);
    r.n = __shfl(vn0, r.b, 64) - r.n0;
  } else {
    r.n0 = a.node_off[r.b];
    r.n = a.node_off[r.b + 1] - r.n0;
  }
  if (!r.ok) r.n0 = r.n = 0;
  return r;
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
// parents, tokens and tags are already in LDS; its predicate bits and argmaxes
// (written by the other row workgroups) are read once with device-coherent
// loads.  Every lane walks its leaves' chains once (recording the chain in
// LDS), so no chain step touches global memory.
__device__ void path_reduce(const VocabArgs& a, int b, int n0, int n, int L, const int* s_par, const int* s_tok,
                            const uint8_t* s_src, uint8_t* s_flag, uint8_t* s_hc, int* s_am, uint8_t* s_chain,
                            int lane) {
  bool bad_tree = false, bad_tok = false;
  for (int j = lane; j < n; j += 64) {
    const int p = s_par[j];
    s_flag[j] = (uint8_t)ld_dev(a.flag_ws + n0 + j);
    s_am[j] = ld_dev(a.argmax + n0 + j);
    s_hc[j] = 0;
    if (j == 0) {
      bad_tree |= p != -1;
    } else {
      bad_tree |= p < 0 || p >= j;
      const int t = s_tok[j];
      bad_tok |= t < 0 || t >= a.vocab || s_src[j] > 1;
    }
  }
  bad_tree = __any(bad_tree);
  bad_tok = __any(bad_tok);
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
struct FinalizeLds {
  float st[4][4];
  uint64_t key[4][KO];
  float row[4];         // m, lse, -, argmax of the row (after the merge)
  uint64_t top[KO];     // the row's top-K keys
  int par[kMaxNodes];
  int tok[kMaxNodes];
  uint8_t src[kMaxNodes];
  int node_am[kMaxNodes];
  uint8_t flag[kMaxNodes];
  uint8_t hc[kMaxNodes];
  uint8_t chain[64 * kMaxDepth];
  int ticket;
};

// One node row: statistics, children's predicates, and (last row of the
// sequence) the path.  Wide: batch >= 64 (node offsets in several groups).
template <int KO, bool Wide>
__device__ __forceinline__ void finalize_row(const VocabArgs& a, FinalizeLds<KO>& sh) {
  constexpr int W = TilePartial<KO>::kWords;
  constexpr int kLoadBatch = 2;  // tile partials per thread requested up front
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int tid = threadIdx.x;
  const int i = blockIdx.x;

  // Requests, in the order their data is needed later: the node offsets, this
  // thread's tile partials, then (once the sequence is known) one node's
  // parent, token and tag per thread.  All are issued by every lane with
  // clamped indices, so the load counts are the same on every path.
  const uint32_t* prow = reinterpret_cast<const uint32_t*>(a.partials) + (size_t)i * a.n_vtiles * W;
  u32x4 buf[kLoadBatch][W / 4];
  int v0, vn0;
  load_offsets(a, lane, v0, vn0);
#pragma unroll
  for (int u = 0; u < kLoadBatch; ++u) {
    const int t = min(tid + u * (int)blockDim.x, a.n_vtiles - 1);
#pragma unroll
    for (int q = 0; q < W / 4; ++q) buf[u][q] = *reinterpret_cast<const u32x4*>(prow + (size_t)t * W + 4 * q);
  }
  const SeqLayout lay = scan_layout<Wide>(a, i, lane, v0, vn0);
  const bool lay_ok = lay.ok;
  const int b = lay.b, n0 = lay.n0, n = lay.n;
  const int li = i - n0;
  const int jn = lay_ok ? n0 + min(tid, n - 1) : 0;
  const int c_par = a.parent[jn];
  const int c_tok = a.token[jn];
  const int c_src = a.src[jn];

  // fold the row's tile partials: this thread's tiles, then the wave
  RowStats st;
  st.init();
  uint64_t key[KO];
#pragma unroll
  for (int k = 0; k < KO; ++k) key[k] = 0ull;
  auto fold = [&](const u32x4 (&pb)[W / 4]) {
    st.merge(__uint_as_float(pb[0][0]), __uint_as_float(pb[0][1]), __uint_as_float(pb[0][2]), (int)pb[0][3]);
    uint64_t pk[KO];
#pragma unroll
    for (int k = 0; k < KO; ++k) {
      const u32x4 w4 = pb[1 + k / 2];
      pk[k] = (k & 1) ? (((uint64_t)w4[3] << 32) | w4[2]) : (((uint64_t)w4[1] << 32) | w4[0]);
    }
    merge_topk<KO>(key, pk);
  };
#pragma unroll
  for (int u = 0; u < kLoadBatch; ++u)
    if (tid + u * (int)blockDim.x < a.n_vtiles) fold(buf[u]);
  for (int t = tid + kLoadBatch * blockDim.x; t < a.n_vtiles; t += blockDim.x) {
    u32x4 pb[W / 4];
#pragma unroll
    for (int q = 0; q < W / 4; ++q) pb[q] = *reinterpret_cast<const u32x4*>(prow + (size_t)t * W + 4 * q);
    fold(pb);
  }
  st.merge_level<0>();
  merge_topk_level<KO, 0>(key);
  st.merge_level<1>();
  merge_topk_level<KO, 1>(key);
  st.merge_level<2>();
  merge_topk_level<KO, 2>(key);
  // the children of node li request their logit z_li[t] while the merge goes on
  // (scheduling barriers keep the request here, after the parents have had time to arrive)
  __builtin_amdgcn_sched_barrier(0);
  const bool is_child = lay_ok && tid < n && tid > 0 && c_par == li;
  const bool tok_ok = c_tok >= 0 && c_tok < a.vocab;
  const float c_z = a.logits[(size_t)i * a.vocab + (is_child && tok_ok ? c_tok : 0)];
  __builtin_amdgcn_sched_barrier(0);
  st.merge_level<3>();
  merge_topk_level<KO, 3>(key);
  st.merge_level<4>();
  merge_topk_level<KO, 4>(key);
  st.merge_level<5>();
  merge_topk_level<KO, 5>(key);
  if (lane == 0) {
    sh.st[wave][0] = st.m;
    sh.st[wave][1] = st.S;
    sh.st[wave][2] = st.T;
    sh.st[wave][3] = __int_as_float(st.am);
#pragma unroll
    for (int k = 0; k < KO; ++k) sh.key[wave][k] = key[k];
  }
  if (lay_ok && tid < n) {
    sh.par[tid] = c_par;
    sh.tok[tid] = c_tok;
    sh.src[tid] = (uint8_t)c_src;
  }
  __syncthreads();
  // across the 4 waves (wave 0; lanes of a quad hold the 4 wave results); the
  // row's results go to LDS first and to memory after the barrier, so that the
  // barrier does not wait for the stores
  if (wave == 0) {
    const int src_wave = lane & 3;
    st.m = sh.st[src_wave][0];
    st.S = sh.st[src_wave][1];
    st.T = sh.st[src_wave][2];
    st.am = __float_as_int(sh.st[src_wave][3]);
#pragma unroll
    for (int k = 0; k < KO; ++k) key[k] = sh.key[src_wave][k];
    st.merge_level<0>();
    merge_topk_level<KO, 0>(key);
    st.merge_level<1>();
    merge_topk_level<KO, 1>(key);
    if (lane == 0) {
      sh.row[0] = st.m;
      sh.row[1] = st.m + __logf(st.S);
      sh.row[3] = __int_as_float(st.am);
#pragma unroll
      for (int k = 0; k < KO; ++k) sh.top[k] = key[k];
    }
  }
  __syncthreads();
  if (wave == 0) {
    const float logS = __logf(st.S);
    const float lse = st.m + logS;
    if (lane == 0) {
      a.max_logit[i] = st.m;
      st_dev(a.argmax + i, st.am);
      a.lse[i] = lse;
      a.entropy[i] = logS - st.T / st.S;
    }
#pragma unroll
    for (int k = 0; k < KO; ++k)
      if (lane == k && k < a.topk_out) {
        a.topk_id[(size_t)i * a.topk_out + k] = key_id(key[k]);
        a.topk_logprob[(size_t)i * a.topk_out + k] = key_value(key[k]) - lse;
      }
  }
  if (!lay_ok) return;  // uniform over the workgroup

  // predicates of the children of node li: thread j describes node j
  if (is_child) {
    const float m = sh.row[0], lse = sh.row[1];
    const int am = __float_as_int(sh.row[3]);
    uint32_t f = 0;
    float lp = 0.f;
    if (tok_ok) {
      bool intop = false;
#pragma unroll
      for (int k = 0; k < KO; ++k) intop |= (k < a.topk) && (key_id(sh.top[k]) == c_tok);
      if (c_tok == am) f |= kFlagGreedy;
      if (intop) f |= kFlagTopk;
      if ((double)m - (double)c_z <= (double)a.tau) f |= kFlagTau;
      if (c_src == 1 && (f & kFlagTopk) && (f & kFlagTau)) f |= kFlagRelaxed;
      lp = c_z - lse;
    }
    st_dev(a.flag_ws + n0 + tid, (int32_t)f);
    a.tok_logprob[n0 + tid] = lp;
  }
  if (li == 0 && tid == 0) {
    st_dev(a.flag_ws + n0, 0);
    a.tok_logprob[n0] = 0.f;
  }

  // ---- sequence completion ticket ----
  stores_done();
  __syncthreads();
  if (tid == 0) sh.ticket = atomicAdd(a.seq_counter + b, 1);
  __syncthreads();
  if (sh.ticket != n - 1 || wave != 0) return;
  path_reduce(a, b, n0, n, a.kv_len[b], sh.par, sh.tok, sh.src, sh.flag, sh.hc, sh.node_am, sh.chain, lane);
  if (lane == 0) st_dev(a.seq_counter + b, 0);
}

template <int KO>
__global__ __launch_bounds__(256) void finalize_kernel(VocabArgs a) {
  __shared__ FinalizeLds<KO> sh;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (blockIdx.x >= (unsigned)a.total_nodes) {
    // sequence report: only sequences that no row workgroup can finish
    const int b = blockIdx.x - a.total_nodes;
    if (wave != 0) return;
    int v0, vn0;
    load_offsets(a, lane, v0, vn0);
    const SeqLayout lay = a.batch < 64 ? scan_layout<false>(a, 0, lane, v0, vn0) : scan_layout<true>(a, 0, lane, v0, vn0);
    if (b >= a.batch || lay.ok) return;
    write_seq_error(a, b, kStatusTree, 0, 0, lane);
    return;
  }
  if (a.batch < 64)
    finalize_row<KO, false>(a, sh);
  else
    finalize_row<KO, true>(a, sh);
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
