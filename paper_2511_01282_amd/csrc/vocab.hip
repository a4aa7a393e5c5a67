// Row finalisation and path reduction of a draft-tree verification step.
//
// Per node row i (ReSpec: entropy of Eq. 1; relaxed check of Eq. 6-7;
// look-ahead tolerance of Section 3.4; winner of Algorithm 1's RelaxedVerify):
//   1. one workgroup merges the row's per-tile statistics written by the
//      LM-head epilogue (online max / sum / entropy terms and the tile's
//      (max, argmax)): lse = m + log S, entropy = log S - T/S; the row's top-K
//      entries lie in the tiles with the K largest maxima, so only those are
//      read back to give the exact top-k by (z desc, id asc); then, for every
//      child j of node i, the predicates of
//      j's token: GREEDY (t == argmax), TOPK (t among the first k), TAU
//      (z_max - z_t <= tau, compared in double), RELAXED (retrieved and TOPK and
//      TAU);
//   2. the last row of a sequence to finish (device-scope ticket; predicates
//      handed over with device-coherent stores and loads) runs the look-ahead
//      procedure on every root-to-leaf chain (64-bit chain masks, one lane per
//      leaf) and picks the winner: longest accepted length, then smallest last
//      accepted node, then smallest leaf.  Every row checks the sequence's tree
//      and walks its leaf chains before taking the ticket (that needs only the
//      parents), so the winner of the ticket only reads the predicates.
// A row is reduced by four waves (one when the vocabulary has at most 64
// tiles): each wave reduces its lanes' statistics by wave-wide reductions,
// picks its K largest tile maxima by repeated maxima, reads those tiles and
// takes their top-K the same way; then wave 0 combines the waves.
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

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t x) {
  uint64_t y;
  y = xchg<0>(x); x = y > x ? y : x;
  y = xchg<1>(x); x = y > x ? y : x;
  y = xchg<2>(x); x = y > x ? y : x;
  y = xchg<3>(x); x = y > x ? y : x;
  y = xchg<4>(x); x = y > x ? y : x;
  y = xchg<5>(x); x = y > x ? y : x;
  return x;
}

// Top K keys of a wave whose lanes each hold a descending list of L keys:
// K rounds of "wave maximum of the lanes' heads, whose owner pops it".  Keys
// are distinct (the low word holds the token id) or 0 (empty slot).  Every
// lane receives the same top[].
template <int L, int K>
__device__ __forceinline__ void wave_topk(uint64_t (&key)[L], uint64_t (&top)[K]) {
#pragma unroll
  for (int r = 0; r < K; ++r) {
    const uint64_t mx = wave_max_u64(key[0]);
    top[r] = mx;
    const bool pop = key[0] == mx;
#pragma unroll
    for (int k = 0; k + 1 < L; ++k) key[k] = pop ? key[k + 1] : key[k];
    key[L - 1] = pop ? 0ull : key[L - 1];
  }
}

// Descending sort of a thread's N keys (bitonic network, N a power of two).
template <int N>
__device__ __forceinline__ void sort_desc(uint64_t (&k)[N]) {
#pragma unroll
  for (int sz = 2; sz <= N; sz *= 2)
#pragma unroll
    for (int j = sz / 2; j > 0; j /= 2)
#pragma unroll
      for (int x = 0; x < N; ++x) {
        const int y = x ^ j;
        if (y > x) {
          const bool desc = (x & sz) == 0;  // the last stage (sz = N) sorts all of it descending
          const bool sw = desc ? k[y] > k[x] : k[x] > k[y];
          const uint64_t kx = k[x], ky = k[y];
          k[x] = sw ? ky : kx;
          k[y] = sw ? kx : ky;
        }
      }
}

// Insert key v into a descending list of N keys, dropping the smallest.
template <int N>
__device__ __forceinline__ void insert_desc(uint64_t (&k)[N], uint64_t v) {
#pragma unroll
  for (int x = N - 1; x > 0; --x) k[x] = v > k[x - 1] ? k[x - 1] : (v > k[x] ? v : k[x]);
  k[0] = v > k[0] ? v : k[0];
}

// Value held by lane (lane ^ J), J a power of two up to 32: DPP row moves
// give xor 1 and xor 2; xor 4 is xor 3 (quad reversal) followed by the mirror
// within 8 (xor 7), xor 8 the mirror within 8 followed by the mirror within 16
// (xor 15); xor 16 and 32 are the row swaps.
template <int J>
__device__ __forceinline__ int lane_xor(int v) {
  if constexpr (J == 1) return xchg<0>(v);
  if constexpr (J == 2) return xchg<1>(v);
  if constexpr (J == 4) return xchg<2>(__builtin_amdgcn_mov_dpp(v, 0x1B, 0xF, 0xF, false));  // quad_perm 3,2,1,0
  if constexpr (J == 8) return xchg<3>(xchg<2>(v));
  if constexpr (J == 16) return xchg<4>(v);
  return xchg<5>(v);
}
template <int J>
__device__ __forceinline__ uint64_t lane_xor(uint64_t v) {
  const uint32_t lo = (uint32_t)lane_xor<J>((int)(uint32_t)v), hi = (uint32_t)lane_xor<J>((int)(uint32_t)(v >> 32));
  return ((uint64_t)hi << 32) | lo;
}

// One compare-exchange stage of a bitonic network over the 64 lanes: blocks
// of S lanes, partner lane ^ J; a block is ordered descending when lane & S
// is 0, so the last stages (S = 64) order the whole wave descending.
template <int S, int J>
__device__ __forceinline__ uint64_t bitonic_stage(uint64_t k, int lane) {
  const uint64_t o = lane_xor<J>(k);
  const bool desc = (lane & S) == 0;
  const bool keep_max = ((lane & J) == 0) == desc;
  const uint64_t mx = o > k ? o : k, mn = o > k ? k : o;
  return keep_max ? mx : mn;
}

// Sort one key per lane across the wave, descending: lane 0 receives the
// largest (21 compare-exchange stages).
__device__ __forceinline__ uint64_t wave_sort_desc(uint64_t k) {
  const int lane = (int)(threadIdx.x & 63);
  k = bitonic_stage<2, 1>(k, lane);
  k = bitonic_stage<4, 2>(k, lane);
  k = bitonic_stage<4, 1>(k, lane);
  k = bitonic_stage<8, 4>(k, lane);
  k = bitonic_stage<8, 2>(k, lane);
  k = bitonic_stage<8, 1>(k, lane);
  k = bitonic_stage<16, 8>(k, lane);
  k = bitonic_stage<16, 4>(k, lane);
  k = bitonic_stage<16, 2>(k, lane);
  k = bitonic_stage<16, 1>(k, lane);
  k = bitonic_stage<32, 16>(k, lane);
  k = bitonic_stage<32, 8>(k, lane);
  k = bitonic_stage<32, 4>(k, lane);
  k = bitonic_stage<32, 2>(k, lane);
  k = bitonic_stage<32, 1>(k, lane);
  k = bitonic_stage<64, 32>(k, lane);
  k = bitonic_stage<64, 16>(k, lane);
  k = bitonic_stage<64, 8>(k, lane);
  k = bitonic_stage<64, 4>(k, lane);
  k = bitonic_stage<64, 2>(k, lane);
  k = bitonic_stage<64, 1>(k, lane);
  return k;
}

__device__ __forceinline__ uint64_t readlane64(uint64_t v, int l) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), l);
  return ((uint64_t)hi << 32) | lo;
}

// Append, in lane order, the values of the lanes with take set to a wave's
// LDS list of capacity cap; count (the same in every lane) grows by their
// number, also past cap (entries past cap are not written).
template <typename T>
__device__ __forceinline__ void wave_append(T* list, int& count, bool take, T v, int cap) {
  const uint64_t bal = __ballot(take);
  const int pos = count + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32),
                                                         __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u));
  if (take && pos < cap) list[pos] = v;
  count += __popcll(bal);
}

// Softmax statistics of the wave's union of disjoint sets: the maximum first,
// then every lane's sums rescaled to it (T = sum e^(z-M) (z-M)) and added; the
// argmax is the smallest id among lanes at the maximum.
__device__ __forceinline__ void wave_rowstats(RowStats& st) {
  float M = st.m;
  M = fmaxf(M, xchg<0>(M));
  M = fmaxf(M, xchg<1>(M));
  M = fmaxf(M, xchg<2>(M));
  M = fmaxf(M, xchg<3>(M));
  M = fmaxf(M, xchg<4>(M));
  M = fmaxf(M, xchg<5>(M));
  const bool empty = st.m == -__builtin_huge_valf();
  const float d = empty ? 0.f : st.m - M;
  const float e = empty ? 0.f : __expf(d);
  float S = st.S * e, T = (st.T + d * st.S) * e;
  int am = (!empty && st.m == M) ? st.am : 0x7FFFFFFF;
  S += xchg<0>(S); T += xchg<0>(T); am = min(am, xchg<0>(am));
  S += xchg<1>(S); T += xchg<1>(T); am = min(am, xchg<1>(am));
  S += xchg<2>(S); T += xchg<2>(T); am = min(am, xchg<2>(am));
  S += xchg<3>(S); T += xchg<3>(T); am = min(am, xchg<3>(am));
  S += xchg<4>(S); T += xchg<4>(T); am = min(am, xchg<4>(am));
  S += xchg<5>(S); T += xchg<5>(T); am = min(am, xchg<5>(am));
  st.m = M;
  st.S = S;
  st.T = T;
  st.am = am;
}

// Look-ahead tolerance on one chain u_1..u_d; bit s-1 of G / OK describes u_s
// (no bits at or above d).  Runs of greedy matches are counted with
// count-trailing-zeros of the complement.
__device__ __forceinline__ int ones_from(uint64_t G, int s) {  // consecutive set bits of G from bit s up
  if (s >= 64) return 0;
  const uint64_t z = ~(G >> s);
  return z == 0 ? 64 - s : __builtin_ctzll(z);
}

__device__ __forceinline__ int lookahead_bits(int d, uint64_t G, uint64_t OK, int m, int phi) {
  const int l0 = ones_from(G, 0);
  int cur = l0, last = l0;
  for (int att = 0; att < phi && cur < d; ++att) {
    if (!((OK >> cur) & 1ull)) break;
    const int xi = ones_from(G, cur + 1);
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

// Chains of the leaves of one sequence, walked once per row workgroup before
// the completion ticket (they need only the parents, which every row holds in
// LDS).  Lane l owns leaves l and l + 64; chain[it][l][k] is the node k steps
// above leaf l + 64*it (the leaf itself at k = 0), depth[it] its depth, or -1
// for a node with children.
struct PathPrep {
  int depth[2];
  bool bad_tree, bad_tok, too_deep;
};

__device__ __forceinline__ PathPrep path_prepare(const VocabArgs& a, int n, const int* s_par, const int* s_tok,
                                                 const uint8_t* s_src, uint8_t* s_hc, uint8_t* s_chain, int lane) {
  PathPrep pp{{-1, -1}, false, false, false};
  bool bad_tree = false, bad_tok = false;
  for (int j = lane; j < n; j += 64) {
    const int p = s_par[j];
    s_hc[j] = 0;
    if (j == 0) {
      bad_tree |= p != -1;
    } else {
      bad_tree |= p < 0 || p >= j;
      const int t = s_tok[j];
      bad_tok |= t < 0 || t >= a.vocab || s_src[j] > 1;
    }
  }
  pp.bad_tree = __any(bad_tree);
  pp.bad_tok = __any(bad_tok);
  if (pp.bad_tree) return pp;
  wave_lds_sync();
  for (int j = lane; j < n; j += 64)
    if (j > 0) s_hc[s_par[j]] = 1;
  wave_lds_sync();
  // parents strictly decrease, so every walk ends at the root within n steps
  bool too_deep = false;
#pragma unroll
  for (int it = 0; it < 2; ++it) {
    const int j = lane + 64 * it;
    if (j >= n || s_hc[j]) continue;
    uint8_t* chain = s_chain + (it * 64 + lane) * kMaxDepth;
    int d = 0, x = j;
    while (x != 0 && d < kMaxDepth) {
      chain[d] = (uint8_t)x;
      x = s_par[x];
      ++d;
    }
    if (x != 0 || d > a.max_depth) {
      too_deep = true;
      continue;
    }
    pp.depth[it] = d;
  }
  pp.too_deep = __any(too_deep);
  return pp;
}

// One wave, after winning the sequence's ticket: read every node's predicate
// bits and argmax (written by the other rows), run the look-ahead procedure on
// the chains prepared above, and write the winner, its path and the flags.
__device__ void path_finish(const VocabArgs& a, int b, int n0, int n, int L, const PathPrep& pp, const int* s_par,
                            uint8_t* s_flag, int* s_am, const uint8_t* s_chain, int lane) {
  const bool bad_cap = L < 0 || L > a.max_kv || L > a.kv_cap - n;
  const bool bad_tree = pp.bad_tree || pp.too_deep;
  const int status = bad_tree ? kStatusTree : pp.bad_tok ? kStatusToken : bad_cap ? kStatusCapacity : 0;
  if (status != 0) {
    write_seq_error(a, b, status, n0, n, lane);
    return;
  }
  for (int j = lane; j < n; j += 64) {
    s_flag[j] = (uint8_t)ld_dev(a.flag_ws + n0 + j);
    s_am[j] = ld_dev(a.argmax + n0 + j);
  }
  wave_lds_sync();
  uint64_t best = ~0ull;
#pragma unroll
  for (int it = 0; it < 2; ++it) {
    const int j = lane + 64 * it;
    if (j >= n) continue;
    const int d = pp.depth[it];
    if (d < 0) {
      a.leaf_acc_len[n0 + j] = -1;
      continue;
    }
    const uint8_t* chain = s_chain + (it * 64 + lane) * kMaxDepth;
    uint64_t G = 0, OK = 0;  // bit s-1 describes u_s, the node at depth s (chain[d - s])
    for (int k0 = 0; k0 < d; k0 += 8) {
      const uint64_t c8 = *reinterpret_cast<const uint64_t*>(chain + k0);  // 8 chain entries at once
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int k = k0 + u;
        const uint32_t f = k < d ? s_flag[(c8 >> (8 * u)) & 0xFFu] : 0u;
        const int bit = d - 1 - k;
        G |= k < d ? (uint64_t)(f & kFlagGreedy) << bit : 0ull;
        OK |= k < d ? (uint64_t)((f & (kFlagGreedy | kFlagRelaxed)) != 0) << bit : 0ull;
      }
    }
    const int acc = lookahead_bits(d, G, OK, a.min_lookahead, a.max_relaxed);
    const int e = acc == 0 ? 0 : chain[d - acc];
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

constexpr int kMaxCandTiles = 256;  // >= K * (tile keys per thread)

template <int KO>
struct FinalizeLds {
  float st[4][4];
  uint64_t key[4][KO];
  float row[4];         // m, lse, -, argmax of the row (after the merge)
  uint64_t top[KO];     // the row's top-K keys
  int ctile[4][kMaxCandTiles];  // per wave: candidate tiles
  uint64_t surv[4][64];         // per wave: candidate logits that reach the threshold
  int par[kMaxNodes];
  int tok[kMaxNodes];
  uint8_t src[kMaxNodes];
  int node_am[kMaxNodes];
  uint8_t flag[kMaxNodes];
  uint8_t hc[kMaxNodes];
  alignas(8) uint8_t chain[2 * 64 * kMaxDepth];
  int ticket;
};

// One node row: statistics, children's predicates, and (last row of the
// sequence) the path.  WPR waves reduce the row (1 or 4); each thread keeps
// the keys of up to LB tiles.  Wide: batch >= 64 (node offsets in several
// groups).
template <int KO, int WPR, int LB, bool Wide>
__device__ __forceinline__ void finalize_row(const VocabArgs& a, FinalizeLds<KO>& sh) {
  constexpr int NT = 64 * WPR;   // threads of the row
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int tid = threadIdx.x;
  const int i = blockIdx.x;

  // Requests, in the order their data is needed later: the node offsets, this
  // thread's tile partials, then (once the sequence is known) the parent, token
  // and tag of nodes tid and tid + NT.  All are issued by every lane with
  // clamped indices, so the load counts are the same on every path.
  const u32x4* prow = reinterpret_cast<const u32x4*>(a.partials) + (size_t)i * a.n_vtiles;
  u32x4 buf[LB];
  int v0, vn0;
  load_offsets(a, lane, v0, vn0);
#pragma unroll
  for (int u = 0; u < LB; ++u) {
    const int t = min(tid + u * NT, a.n_vtiles - 1);
    buf[u] = prow[t];
  }
  const SeqLayout lay = scan_layout<Wide>(a, i, lane, v0, vn0);
  const bool lay_ok = lay.ok;
  const int b = lay.b, n0 = lay.n0, n = lay.n;
  const int li = i - n0;
  constexpr int NPT = (kMaxNodes + NT - 1) / NT;  // nodes described per thread
  int c_par[NPT], c_tok[NPT], c_src[NPT];
#pragma unroll
  for (int u = 0; u < NPT; ++u) {
    const int jn = lay_ok ? n0 + min(tid + u * NT, n - 1) : 0;
    c_par[u] = a.parent[jn];
    c_tok[u] = a.token[jn];
    c_src[u] = a.src[jn];
  }
  const int kv_b = a.kv_len[lay_ok ? b : 0];
  // node i's own parent and token: the rank pass counts node i's token in its parent's row
  int my_par = -1, my_tok = -1;
  if (a.rank_req) {
    my_par = a.parent[i];
    my_tok = a.token[i];
  }

  // Fold the row's tile statistics (this thread's tiles), and keep each tile's
  // largest (value, id) key; the id's tile is the tile.
  RowStats st;
  st.init();
  uint64_t tk[LB];  // this thread's tile keys, descending after the sort below
#pragma unroll
  for (int u = 0; u < LB; ++u) {
    const bool ok = tid + u * NT < a.n_vtiles;
    const float m_t = __uint_as_float(buf[u][0]);
    const int am_t = (int)buf[u][3];
    if (ok) st.merge(m_t, __uint_as_float(buf[u][1]), __uint_as_float(buf[u][2]), am_t);
    tk[u] = ok ? make_key(m_t, am_t) : 0ull;
  }
  const bool spill = a.n_vtiles > LB * NT;  // (uniform) tiles past the key lists: read the whole row
  for (int t = tid + LB * NT; t < a.n_vtiles; t += NT) {
    const u32x4 pb = prow[t];
    st.merge(__uint_as_float(pb[0]), __uint_as_float(pb[1]), __uint_as_float(pb[2]), (int)pb[3]);
  }
  // Candidate tiles of this wave.  H, the K-th largest of the lanes' largest
  // tile keys, is the smallest of K distinct tile maxima, so the wave's K-th
  // largest logit key is at least H: every entry of the row's top-K that lies
  // in this wave's tiles has a key >= H and lies in a tile whose maximum key
  // is >= H (at most K lanes hold such tiles).
  uint64_t head = tk[0];
#pragma unroll
  for (int u = 1; u < LB; ++u) head = tk[u] > head ? tk[u] : head;
  const uint64_t H = readlane64(wave_sort_desc(head), KO - 1);  // 0: fewer than K tiles
  int* ct = sh.ctile[wave];
  int nt = 0;
#pragma unroll
  for (int u = 0; u < LB; ++u) {
    const uint32_t t = (uint32_t)key_id(tk[u]) / kLmTileRows;  // the tile of its maximum
    wave_append(ct, nt, tk[u] != 0 && tk[u] >= H && t < (uint32_t)a.n_vtiles, (int)t, kMaxCandTiles);
  }
  // the children of node li request their logit z_li[t] now (the parents have had time to arrive)
  bool is_child[NPT], tok_ok[NPT];
  float c_z[NPT];
#pragma unroll
  for (int u = 0; u < NPT; ++u) {
    const int j = tid + u * NT;
    is_child[u] = lay_ok && j < n && j > 0 && c_par[u] == li;
    tok_ok[u] = c_tok[u] >= 0 && c_tok[u] < a.vocab;
    c_z[u] = a.logits[(size_t)i * a.vocab + (is_child[u] && tok_ok[u] ? c_tok[u] : 0)];
  }
  wave_lds_sync();
  // The candidates' logits (8 tiles per pass: 8 lanes per tile, 8 columns
  // each); those with a key >= H go to the wave's survivor list.
  const float* zrow = a.logits + (size_t)i * a.vocab;
  uint64_t* sv = sh.surv[wave];
  int nv = 0;
  // More candidate tiles than the list holds only happens when tile keys repeat,
  // which statistics written by the LM head never do (a tile's argmax lies in
  // that tile); the wave then reads all of its own tiles instead, and never
  // indexes past the list.
  const bool cand_over = nt > kMaxCandTiles;  // (uniform over the wave)
  nt = min(nt, kMaxCandTiles);
  auto cand_pass = [&](int p0, uint64_t (&kz)[8]) {
    const int c = p0 + (lane >> 3);
    const int col0 = c < nt ? ct[c] * kLmTileRows + (lane & 7) : a.vocab;
    float z[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) z[e] = col0 + 8 * e < a.vocab ? zrow[col0 + 8 * e] : 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint64_t kv = col0 + 8 * e < a.vocab ? make_key(z[e], col0 + 8 * e) : 0ull;
      kz[e] = kv != 0 && kv >= H ? kv : 0ull;
    }
  };
  if (!spill && !cand_over) {
    for (int p0 = 0; p0 < nt; p0 += 8) {
      uint64_t kz[8];
      cand_pass(p0, kz);
#pragma unroll
      for (int e = 0; e < 8; ++e) wave_append(sv, nv, kz[e] != 0, kz[e], 64);
    }
  }
  // the sequence's nodes go to LDS (the path reduction reads them)
  if (lay_ok) {
#pragma unroll
    for (int u = 0; u < NPT; ++u) {
      const int j = tid + u * NT;
      if (j < n) {
        sh.par[j] = c_par[u];
        sh.tok[j] = c_tok[u];
        sh.src[j] = (uint8_t)c_src[u];
      }
    }
  }
  // the wave's statistics (by reductions)
  wave_rowstats(st);
  if constexpr (WPR > 1) {
    if (lane == 0) {
      sh.st[wave][0] = st.m;
      sh.st[wave][1] = st.S;
      sh.st[wave][2] = st.T;
      sh.st[wave][3] = __int_as_float(st.am);
    }
  }
  wave_lds_sync();
  // The wave's top-K: lane k < K receives the k-th key.  Normally at most 64
  // survivors, sorted across the wave; otherwise (many equal values, or rows
  // read whole) per-lane top-K lists and K rounds of wave maxima.
  uint64_t kk;
  if (!spill && !cand_over && nv <= 64) {
    kk = wave_sort_desc(lane < nv ? sv[lane] : 0ull);
  } else {
    uint64_t ck[KO];
#pragma unroll
    for (int k = 0; k < KO; ++k) ck[k] = 0ull;
    if (!spill && !cand_over) {
      for (int p0 = 0; p0 < nt; p0 += 8) {
        uint64_t kz[8];
        cand_pass(p0, kz);
#pragma unroll
        for (int e = 0; e < 8; ++e) insert_desc<KO>(ck, kz[e]);
      }
    } else if (!spill) {  // every column of this thread's own tiles
#pragma unroll
      for (int u = 0; u < LB; ++u) {
        const int t = tid + u * NT;
        if (t >= a.n_vtiles) continue;
        for (int e = 0; e < kLmTileRows; ++e) {
          const int col = t * kLmTileRows + e;
          if (col < a.vocab) insert_desc<KO>(ck, make_key(zrow[col], col));
        }
      }
    } else {
      for (int col = tid; col < a.vocab; col += NT) insert_desc<KO>(ck, make_key(zrow[col], col));
    }
    uint64_t top[KO];
    wave_topk<KO, KO>(ck, top);
    kk = 0ull;
#pragma unroll
    for (int k = 0; k < KO; ++k) kk = lane == k ? top[k] : kk;
  }
  if constexpr (WPR > 1) {
    if (lane < KO) sh.key[wave][lane] = kk;
    __syncthreads();
    // across the waves (wave 0): lane w < WPR brings wave w's statistics, lane
    // l < WPR*K one key of wave l / K's list
    if (wave == 0) {
      const bool src_ok = lane < WPR;
      st.m = src_ok ? sh.st[lane][0] : -__builtin_huge_valf();
      st.S = src_ok ? sh.st[lane][1] : 0.f;
      st.T = src_ok ? sh.st[lane][2] : 0.f;
      st.am = src_ok ? __float_as_int(sh.st[lane][3]) : 0x7FFFFFFF;
      wave_rowstats(st);
      kk = wave_sort_desc(lane < WPR * KO ? sh.key[lane / KO][lane % KO] : 0ull);
    }
  }
  // row results: LDS for the predicates, memory for the outputs (wave 0)
  if (wave == 0) {
    const float logS = __logf(st.S);
    const float lse = st.m + logS;
    if (lane == 0) {
      sh.row[0] = st.m;
      sh.row[1] = lse;
      sh.row[3] = __int_as_float(st.am);
      a.max_logit[i] = st.m;
      st_dev(a.argmax + i, st.am);
      a.lse[i] = lse;
      a.entropy[i] = logS - st.T / st.S;
    }
    if (lane < KO) sh.top[lane] = kk;
    if (lane < a.topk_out) {
      a.topk_id[(size_t)i * a.topk_out + lane] = key_id(kk);
      a.topk_logprob[(size_t)i * a.topk_out + lane] = key_value(kk) - lse;
    }
  }
  if constexpr (WPR > 1)
    __syncthreads();
  else
    wave_lds_sync();
  if (a.rank_req && tid == 0) {
    const bool rq = lay_ok && li > 0 && my_par >= 0 && my_par < li && my_tok >= 0 && my_tok < a.vocab;
    a.rank_req[i] = rq ? n0 + my_par : -1;
    a.tok_rank[i] = rq ? 0 : -1;
  }
  if (!lay_ok) return;  // uniform over the workgroup

  // predicates of the children of node li: thread j describes node j (and j + NT)
#pragma unroll
  for (int u = 0; u < NPT; ++u) {
    if (!is_child[u]) continue;
    const int j = tid + u * NT;
    const float m = sh.row[0], lse = sh.row[1];
    const int am = __float_as_int(sh.row[3]);
    uint32_t f = 0;
    float lp = 0.f;
    if (tok_ok[u]) {
      bool intop = false;
#pragma unroll
      for (int k = 0; k < KO; ++k) intop |= (k < a.topk) && (key_id(sh.top[k]) == c_tok[u]);
      if (c_tok[u] == am) f |= kFlagGreedy;
      if (intop) f |= kFlagTopk;
      if ((double)m - (double)c_z[u] <= (double)a.tau) f |= kFlagTau;
      if (c_src[u] == 1 && (f & kFlagTopk) && (f & kFlagTau)) f |= kFlagRelaxed;
      lp = c_z[u] - lse;
    }
    st_dev(a.flag_ws + n0 + j, (int32_t)f);
    a.tok_logprob[n0 + j] = lp;
    if (a.stats_only) a.flags[n0 + j] = (uint8_t)f;
  }
  if (li == 0 && tid == 0) {
    st_dev(a.flag_ws + n0, 0);
    a.tok_logprob[n0] = 0.f;
    if (a.stats_only) a.flags[n0] = 0;
  }
  if (a.stats_only) return;  // (uniform) statistics and predicates only

  // tree checks and leaf chains (wave 0) while the stores drain
  PathPrep pp{};
  if (wave == 0) pp = path_prepare(a, n, sh.par, sh.tok, sh.src, sh.hc, sh.chain, lane);

  // ---- sequence completion ticket ----
  // Every wave's hand-off stores are complete before the workgroup barrier; the
  // ticket is an agent-scope release RMW (it orders them before the count), and
  // the winner, which reads the count of every other row, takes an agent-scope
  // acquire before it reads their hand-off words.
  stores_done();
  if constexpr (WPR > 1) __syncthreads();
  if (tid == 0) sh.ticket = ticket_release(a.seq_counter + b);
  if constexpr (WPR > 1)
    __syncthreads();
  else
    wave_lds_sync();
  if (sh.ticket != n - 1 || wave != 0) return;
  acquire_agent();
  path_finish(a, b, n0, n, kv_b, pp, sh.par, sh.flag, sh.node_am, sh.chain, lane);
  if (lane == 0) st_dev(a.seq_counter + b, 0);
}

template <int KO, int WPR, int LB>
__global__ __launch_bounds__(64 * WPR) void finalize_kernel(VocabArgs a) {
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
    finalize_row<KO, WPR, LB, false>(a, sh);
  else
    finalize_row<KO, WPR, LB, true>(a, sh);
}

template <int KO>
hipError_t launch_finalize_ko(int blocks, const VocabArgs& a, hipStream_t s, hipEvent_t ev_stop) {
  // one wave per row up to 64 vocabulary tiles, else four, with the smallest
  // per-thread key list that holds every tile (beyond 4096 tiles the rows are
  // read whole)
  if (a.n_vtiles <= 64) return launch_k(finalize_kernel<KO, 1, 1>, dim3(blocks), dim3(64), 0, s, nullptr, ev_stop, a);
  if (a.n_vtiles <= 512) return launch_k(finalize_kernel<KO, 4, 2>, dim3(blocks), dim3(256), 0, s, nullptr, ev_stop, a);
  if (a.n_vtiles <= 2048) return launch_k(finalize_kernel<KO, 4, 8>, dim3(blocks), dim3(256), 0, s, nullptr, ev_stop, a);
  return launch_k(finalize_kernel<KO, 4, 16>, dim3(blocks), dim3(256), 0, s, nullptr, ev_stop, a);
}

hipError_t launch_finalize(int ko, int blocks, const VocabArgs& a, hipStream_t s, hipEvent_t ev_stop) {
  if (ko == 8) return launch_finalize_ko<8>(blocks, a, s, ev_stop);
  if (ko == 16) return launch_finalize_ko<16>(blocks, a, s, ev_stop);
  return hipErrorInvalidValue;
}

// Exact rank of node j's token t in its parent's logit row z (float32, as the
// vocabulary pass leaves them): #{u : z_u > z_t} + #{u < t : z_u == z_t}.
// Workgroup (c, j) counts over tokens [c*kRankChunk, (c+1)*kRankChunk) and adds
// its count to tok_rank[j] (zeroed by the vocabulary pass when j has a request).
__global__ __launch_bounds__(256) void rank_kernel(RankArgs a) {
  const int j = blockIdx.y;
  const int row = a.rank_req[j];  // (uniform) parent row, or -1: no rank for node j
  if (row < 0 || row >= a.total_nodes) return;
  const int t = a.token[j];
  if (t < 0 || t >= a.vocab) return;
  const float* zr = a.logits + (size_t)row * a.vocab;
  const float zt = zr[t];
  const int u0 = blockIdx.x * kRankChunk;
  int cnt = 0;
#pragma unroll
  for (int k = 0; k < kRankChunk / 256; ++k) {
    const int u = u0 + k * 256 + (int)threadIdx.x;
    const float z = u < a.vocab ? zr[u] : kNegInf;
    cnt += (u < a.vocab && (z > zt || (z == zt && u < t))) ? 1 : 0;
  }
  for (int o = 32; o > 0; o >>= 1) cnt += __shfl_xor(cnt, o, 64);
  __shared__ int s_cnt[4];
  if ((threadIdx.x & 63) == 0) s_cnt[threadIdx.x >> 6] = cnt;
  __syncthreads();
  if (threadIdx.x == 0) {
    const int total = s_cnt[0] + s_cnt[1] + s_cnt[2] + s_cnt[3];
    if (total) atomicAdd(a.tok_rank + j, total);
  }
}

hipError_t launch_rank(const RankArgs& a, hipStream_t s, hipEvent_t ev_stop) {
  if (a.total_nodes <= 0) return hipSuccess;
  const dim3 grid((a.vocab + kRankChunk - 1) / kRankChunk, a.total_nodes);
  return launch_k(rank_kernel, grid, dim3(256), 0, s, nullptr, ev_stop, a);
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
