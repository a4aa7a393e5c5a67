// Stochastic (lossless) verification of the draft trees (gfx950).
//
// Section 3.4 verifies drafter outputs with standard lossless speculative
// sampling: a draft t drawn from the drafter's distribution q passes with
// probability min(1, p(t)/q(t)) under the target's p = softmax(z / T); after a
// rejection the next token comes from the residual norm(max(p - q, 0)).  A
// tree node tries its children in node order, each against the residual left
// by the rejected ones (recursive rejection over siblings).  A model-drafted
// child uses the drafter's distribution at its parent (draft_prob row); a
// retrieved child is a deterministic draft, q = one-hot at its token.  The
// uniforms are inputs: u[j][0] decides child j, u[j][1] the residual draw at
// node j (inverse CDF over the tokens in increasing order).
//
// One workgroup of 512 threads per node row i (after the vocabulary pass,
// which has written the row's max logit and log-sum-exp):
//   - the residual keeps a closed form: after any sequence of rejections
//     r(v) = [v not in X] * max(p(v) - c * q(v), 0) / N, where X holds the
//     rejected retrieved tokens and c, N are scalars.  Rejecting a retrieved
//     t adds t to X and divides by 1 - r(t) (the mass of every other token);
//     rejecting a model draft sets c <- c + N and multiplies N by the sum of
//     max(p - (c + N) q, 0) over the tokens outside X, one pass over the
//     vocabulary.  So only model rejections and the draw read the row, and a
//     token costs one exponential, one multiply-add and a max.  A pass walks
//     tiles of 2048 tokens, one 16-byte group per thread per tile, with eight
//     tiles' loads in flight per thread (a single workgroup's pass is
//     latency-bound);
//   - the children are tested until one passes; if none does, the residual is
//     drawn in two levels: the same kind of pass leaves each tile's mass in
//     LDS, one wave scans the tile masses to find the tile that holds the
//     threshold, and a block scan inside that tile finds the token;
//   - the row hands its outcome (accepted child, or the draw) to the last row
//     of its sequence (device-scope ticket), which walks the tree from the
//     root along the accepted children and writes the path, the bonus token,
//     the per-leaf accepted lengths and the flags.
#include "../../include/respec_verify.h"
#include "common.hpp"
#include "kernels.hpp"

namespace respec {
namespace {

constexpr int kST = 512;           // threads per row workgroup
constexpr int kSW = kST / 64;      // waves
constexpr int kTile = 4 * kST;     // tokens per tile: one group of 4 per thread
constexpr int kUnroll = 8;         // tiles in flight per thread
constexpr int kMaxTiles = 256;     // vocabularies up to 524288 tokens (checked on the host)
static_assert(kMaxTiles * kTile == kMaxStochVocab, "host limit and LDS table agree");

struct StochLds {
  int par[kMaxNodes];
  int tok[kMaxNodes];
  uint8_t src[kMaxNodes];
  int kid[kMaxNodes];       // children of the row (sequence-local), in node order
  float kz[kMaxNodes];      // z_i[t] and q_i[t] of each child's token (requested together up front)
  float kq[kMaxNodes];
  int excl[kMaxNodes];      // X: rejected retrieved tokens (as child indices)
  uint64_t kids[2];
  float red[kSW];
  float tsum[kMaxTiles][kSW];  // residual mass per tile and wave (the draw)
  int imin[kSW];
  int b, ok;
  int ticket;
  int tile;                 // tile that holds the draw's threshold, -1 past the end
  float tile_pre;           // residual mass before that tile
  float thr;                // the draw's threshold (uniform times the residual mass)
  // the walk (last row of the sequence)
  int nxt[kMaxNodes];
  uint8_t has_child[kMaxNodes];
  uint64_t walked[2];
  int tip, len;
};

__device__ __forceinline__ float block_sum(float v, StochLds& sh, int lane, int wave) {
  v = wave_sum(v);
  if (lane == 0) sh.red[wave] = v;
  __syncthreads();
  float s = 0.f;
#pragma unroll
  for (int w = 0; w < kSW; ++w) s += sh.red[w];
  __syncthreads();
  return s;
}

__device__ __forceinline__ int block_min(int v, StochLds& sh, int lane, int wave) {
  for (int o = 32; o > 0; o >>= 1) v = min(v, __shfl_xor(v, o, 64));
  if (lane == 0) sh.imin[wave] = v;
  __syncthreads();
  int r = sh.imin[0];
#pragma unroll
  for (int w = 1; w < kSW; ++w) r = min(r, sh.imin[w]);
  __syncthreads();
  return r;
}

// Four consecutive values of a row from token v (zeros past the end).  vec:
// the vocabulary is a multiple of 4, so rows are 16-byte aligned.  The loads
// are unconditional (clamped addresses, values masked afterwards): a load
// under a branch would make the compiler wait for every earlier load first.
template <bool Vec>
__device__ __forceinline__ f32x4 load4(const float* row, int v, int V) {
  if constexpr (Vec) {
    const f32x4 x = *reinterpret_cast<const f32x4*>(row + min(v, V - 4));
    const bool in = v < V;
    return f32x4{in ? x.x : 0.f, in ? x.y : 0.f, in ? x.z : 0.f, in ? x.w : 0.f};
  } else {
    const float x0 = row[min(v, V - 1)], x1 = row[min(v + 1, V - 1)], x2 = row[min(v + 2, V - 1)],
                x3 = row[min(v + 3, V - 1)];
    return f32x4{v < V ? x0 : 0.f, v + 1 < V ? x1 : 0.f, v + 2 < V ? x2 : 0.f, v + 3 < V ? x3 : 0.f};
  }
}

struct Row {
  const float* z;
  const float* q;   // null: no model draft rejected or tested yet (or no drafter input)
  int V;
  float m, inv_t, inv_s;
};

// p(v) = softmax(z / T)(v)
__device__ __forceinline__ float target_p(const Row& r, float z) { return __expf((z - r.m) * r.inv_t) * r.inv_s; }

__device__ __forceinline__ bool excluded(const StochLds& sh, int n_excl, int v) {
  bool e = false;
  for (int k = 0; k < n_excl; ++k) e = e || sh.tok[sh.kid[sh.excl[k]]] == v;
  return e;
}

// One pass over the row: thread tid takes tokens 4 * (c * kST + tid) .. +3 of
// every tile c; f(z4, q4, v, c) returns that group's contribution.
template <bool Vec, typename F>
__device__ __forceinline__ float row_pass(const Row& r, int tid, F f) {
  const int n_tiles = (r.V + kTile - 1) / kTile;
  float s = 0.f;
  for (int c0 = 0; c0 < n_tiles; c0 += kUnroll) {
    f32x4 z[kUnroll], q[kUnroll];
    const float* qp = r.q ? r.q : r.z;  // (without a q row the loaded values are unused)
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const int v = 4 * ((c0 + u) * kST + tid);
      z[u] = load4<Vec>(r.z, v, r.V);
      q[u] = load4<Vec>(qp, v, r.V);
    }
    if (!r.q)
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) q[u] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      if (c0 + u < n_tiles) s += f(z[u], q[u], 4 * ((c0 + u) * kST + tid), c0 + u);
    }
  }
  return s;
}

template <bool Vec>
__global__ __launch_bounds__(kST) void stochastic_kernel(StochArgs a) {
  __shared__ StochLds sh;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int i = blockIdx.x;

  // ---- the row's sequence (the layout checks of the vocabulary pass) ----
  if (tid == 0) {
    sh.ok = 1;
    sh.b = 0;
  }
  __syncthreads();
  {
    int before = 0;
    bool bad = false;
    for (int k = tid; k <= a.batch; k += kST) {
      const int v = a.node_off[k];
      const int vn = k < a.batch ? a.node_off[k + 1] : v;
      if (k == 0 && v != 0) bad = true;
      if (k == a.batch && v != a.total_nodes) bad = true;
      if (k < a.batch && (vn - v < 1 || vn - v > a.max_nodes)) bad = true;
      if (k >= 1 && k < a.batch && v <= i) ++before;
    }
    if (bad) sh.ok = 0;
    if (before) atomicAdd(&sh.b, before);
  }
  __syncthreads();
  if (!sh.ok) return;  // the vocabulary pass reported the batch
  const int b = sh.b;
  const int n0 = a.node_off[b], n = a.node_off[b + 1] - n0;
  if (a.seq_status[b] != RESPEC_OK) return;  // tree or token errors: reported already
  const int li = i - n0;

  // ---- tree of the sequence and the row's children ----
  if (tid < n) {
    sh.par[tid] = a.parent[n0 + tid];
    sh.tok[tid] = a.token[n0 + tid];
    sh.src[tid] = a.src[n0 + tid];
  }
  __syncthreads();
  if (wave < 2) {
    const int j = tid;
    const uint64_t mk = __ballot(j < n && j > li && sh.par[j] == li);
    if (lane == 0) sh.kids[wave] = mk;
  }
  __syncthreads();
  const int nk = __popcll(sh.kids[0]) + __popcll(sh.kids[1]);
  if (tid == 0) {
    int c = 0;
    for (int h = 0; h < 2; ++h)
      for (uint64_t mk = sh.kids[h]; mk; mk &= mk - 1) {
        const int j = 64 * h + __builtin_ctzll(mk);
        sh.kid[c] = j;
        ++c;
      }
  }
  __syncthreads();

  Row row;
  row.z = a.logits + (size_t)i * a.vocab;
  row.q = nullptr;
  row.V = a.vocab;
  row.m = a.max_logit[i];
  row.inv_t = a.inv_temp;
  row.inv_s = 1.f;
  const float* qrow = a.draft_prob ? a.draft_prob + (size_t)i * a.vocab : nullptr;
  // every child's z and q at its token, in one round trip (the tests need nothing else per child)
  for (int k = tid; k < nk; k += kST) {
    const int t = sh.tok[sh.kid[k]];
    sh.kz[k] = row.z[t];
    sh.kq[k] = qrow ? qrow[t] : 0.f;
  }
  __syncthreads();

  // ---- p = softmax(z / T): the normaliser ----
  if (a.unit_temp) {
    row.inv_s = __expf(row.m - a.lse[i]);
  } else {
    const float s = row_pass<Vec>(row, tid, [&](f32x4 z, f32x4, int v, int) {
      float t = 0.f;
      t += v < row.V ? __expf((z.x - row.m) * row.inv_t) : 0.f;
      t += v + 1 < row.V ? __expf((z.y - row.m) * row.inv_t) : 0.f;
      t += v + 2 < row.V ? __expf((z.z - row.m) * row.inv_t) : 0.f;
      t += v + 3 < row.V ? __expf((z.w - row.m) * row.inv_t) : 0.f;
      return t;
    });
    row.inv_s = 1.f / block_sum(s, sh, lane, wave);
  }

  // ---- the children, in node order, until one passes ----
  // residual r(v) = [v not in X] * max(p(v) - c q(v), 0) * inv_n
  int accepted = -1, n_excl = 0;
  float c = 0.f, inv_n = 1.f;
  for (int k = 0; k < nk; ++k) {
    const int j = sh.kid[k];
    const int t = sh.tok[j];
    const bool model = qrow && sh.src[j] != RESPEC_SRC_RETRIEVED;
    const float qt_row = sh.kq[k];
    const float rt = excluded(sh, n_excl, t) ? 0.f : fmaxf(target_p(row, sh.kz[k]) - c * qt_row, 0.f) * inv_n;
    const float qt = model ? qt_row : 1.f;
    const float acc = qt > 0.f ? fminf(rt / qt, 1.f) : (rt > 0.f ? 1.f : 0.f);
    if (a.uniform[2 * (size_t)(n0 + j)] < acc) {
      accepted = k;
      break;
    }
    if (!model) {
      // max(r - onehot(t), 0) keeps every other token's mass: normaliser 1 - r(t)
      const float zn = 1.f - rt;
      if (zn > 0.f && rt > 0.f) {
        if (tid == 0) sh.excl[n_excl] = k;
        ++n_excl;
        inv_n /= zn;
        __syncthreads();
      }
      continue;
    }
    // a rejected model draft: sum of max(r - q, 0) = inv_n * sum over v not in X of max(p - (c + N) q, 0)
    row.q = qrow;
    const float c2 = c + 1.f / inv_n;
    float part = row_pass<Vec>(row, tid, [&](f32x4 z, f32x4 q, int v, int) {
      float x = 0.f;
      x += v < row.V ? fmaxf(target_p(row, z.x) - c2 * q.x, 0.f) : 0.f;
      x += v + 1 < row.V ? fmaxf(target_p(row, z.y) - c2 * q.y, 0.f) : 0.f;
      x += v + 2 < row.V ? fmaxf(target_p(row, z.z) - c2 * q.z, 0.f) : 0.f;
      x += v + 3 < row.V ? fmaxf(target_p(row, z.w) - c2 * q.w, 0.f) : 0.f;
      return x;
    });
    for (int e = tid; e < n_excl; e += kST) {
      const int ke = sh.excl[e];
      part -= fmaxf(target_p(row, sh.kz[ke]) - c2 * sh.kq[ke], 0.f);
    }
    const float zn = block_sum(part, sh, lane, wave) * inv_n;
    if (zn > 0.f) {
      c = c2;
      inv_n /= zn;
    }
  }
  const float* q_draw = c > 0.f ? qrow : nullptr;  // q enters the residual only after a model rejection
  row.q = q_draw;

  // ---- no child passed: draw from the residual ----
  int sample = -1;
  if (accepted < 0) {
    const int n_tiles = (row.V + kTile - 1) / kTile;
    // level 1: the mass of max(p - c q, 0) in every tile (and wave), the
    // rejected retrieved tokens taken out afterwards (the common scale inv_n
    // does not change where the threshold falls)
    row_pass<Vec>(row, tid, [&](f32x4 z, f32x4 q, int v, int tile) {
      float x = 0.f;
      x += v < row.V ? fmaxf(target_p(row, z.x) - c * q.x, 0.f) : 0.f;
      x += v + 1 < row.V ? fmaxf(target_p(row, z.y) - c * q.y, 0.f) : 0.f;
      x += v + 2 < row.V ? fmaxf(target_p(row, z.z) - c * q.z, 0.f) : 0.f;
      x += v + 3 < row.V ? fmaxf(target_p(row, z.w) - c * q.w, 0.f) : 0.f;
      x = wave_sum(x);
      if (lane == 0) sh.tsum[tile][wave] = x;
      return 0.f;
    });
    __syncthreads();
    for (int e = tid; e < n_excl; e += kST) {
      const int ke = sh.excl[e];
      const int te = sh.tok[sh.kid[ke]];
      const float x = fmaxf(target_p(row, sh.kz[ke]) - c * (q_draw ? sh.kq[ke] : 0.f), 0.f);
      atomicAdd(&sh.tsum[te / kTile][((te % kTile) / 4) / 64], -x);
    }
    __syncthreads();
    const float u_draw = a.uniform[2 * (size_t)i + 1];
    if (wave == 0) {
      // lane l owns tiles 4l .. 4l+3; tile mass = its waves' sums in wave order
      float tm[4], ls = 0.f;
      int last_tile = -1;
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        const int tc = 4 * lane + h;
        float x = 0.f;
        if (tc < n_tiles)
#pragma unroll
          for (int w = 0; w < kSW; ++w) x += sh.tsum[tc][w];
        x = fmaxf(x, 0.f);
        tm[h] = x;
        ls += x;
        last_tile = x > 0.f ? tc : last_tile;
      }
      float incl = ls;
      for (int o = 1; o < 64; o <<= 1) {
        const float y = __shfl_up(incl, o, 64);
        if (lane >= o) incl += y;
      }
      float excl = __shfl_up(incl, 1, 64);
      if (lane == 0) excl = 0.f;
      const float total = __shfl(incl, 63, 64);
      const float thr = u_draw * total;
      int tile = kMaxTiles;
      float pre = excl;
      if (excl <= thr && thr < incl) {
#pragma unroll
        for (int h = 0; h < 4; ++h) {
          if (tile == kMaxTiles && tm[h] > 0.f && thr < pre + tm[h]) tile = 4 * lane + h;
          if (tile == kMaxTiles) pre += tm[h];
        }
      }
      // the first lane that found a tile; rounding may leave none: then the
      // last tile with mass, searched for its last token with mass
      int best = tile;
      for (int o = 32; o > 0; o >>= 1) best = min(best, __shfl_xor(best, o, 64));
      int lt = last_tile;
      for (int o = 32; o > 0; o >>= 1) lt = max(lt, __shfl_xor(lt, o, 64));
      const int src_lane = best < kMaxTiles ? best / 4 : 0;
      const float best_pre = __shfl(pre, src_lane, 64);
      if (lane == 0) {
        sh.tile = best < kMaxTiles ? best : max(lt, 0);
        sh.tile_pre = best < kMaxTiles ? best_pre : 0.f;
        sh.thr = best < kMaxTiles ? thr : __builtin_inff();
      }
    }
    __syncthreads();
    const int tile = sh.tile;
    const float thr = sh.thr;
    // level 2: the token in the tile whose cumulative mass first exceeds the threshold
    const int v = 4 * (tile * kST + tid);
    const f32x4 z = load4<Vec>(row.z, v, row.V);
    f32x4 q = load4<Vec>(q_draw ? q_draw : row.z, v, row.V);
    if (!q_draw) q = f32x4{0.f, 0.f, 0.f, 0.f};
    const float zz[4] = {z.x, z.y, z.z, z.w};
    const float qq[4] = {q.x, q.y, q.z, q.w};
    float xs[4], own = 0.f;
    int tile_last = -1;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const bool in = v + e < row.V && !excluded(sh, n_excl, v + e);
      xs[e] = in ? fmaxf(target_p(row, zz[e]) - c * qq[e], 0.f) : 0.f;
      own += xs[e];
      tile_last = xs[e] > 0.f ? v + e : tile_last;
    }
    float incl = own;
    for (int o = 1; o < 64; o <<= 1) {
      const float y = __shfl_up(incl, o, 64);
      if (lane >= o) incl += y;
    }
    if (lane == 63) sh.red[wave] = incl;
    __syncthreads();
    float base = sh.tile_pre;
    for (int w = 0; w < wave; ++w) base += sh.red[w];
    float ex = __shfl_up(incl, 1, 64);
    if (lane == 0) ex = 0.f;
    base += ex;
    int found = 0x7fffffff;
    float cum = base;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      cum += xs[e];
      if (found == 0x7fffffff && xs[e] > 0.f && cum > thr) found = v + e;
    }
    __syncthreads();
    const int first = block_min(found, sh, lane, wave);
    const int tl = -block_min(-tile_last, sh, lane, wave);
    sample = max(first != 0x7fffffff ? first : tl, 0);
  }

  // ---- hand-off and the sequence's completion ticket ----
  if (tid == 0) {
    st_dev(a.ws_next + i, accepted >= 0 ? sh.kid[accepted] : -1);
    st_dev(a.ws_sample + i, sample);
    if (a.sample) a.sample[i] = sample;
  }
  stores_done();
  __syncthreads();
  if (tid == 0) sh.ticket = ticket_release(a.seq_counter + b);
  __syncthreads();
  if (sh.ticket != n - 1 || wave != 0) return;
  acquire_agent();  // the other rows' hand-off words are read after their release

  // ---- the walk (one wave, last row of the sequence) ----
  for (int j = lane; j < kMaxNodes; j += 64) {
    sh.has_child[j] = 0;
    sh.nxt[j] = j < n ? ld_dev(a.ws_next + n0 + j) : -1;
  }
  wave_lds_sync();
  for (int j = lane; j < n; j += 64)
    if (j > 0) sh.has_child[sh.par[j]] = 1;
  if (lane == 0) {
    uint64_t w0 = 1ull, w1 = 0ull;
    int cur = 0, len = 0;
    int* prow = a.path + (size_t)b * (a.max_depth + 1);
    prow[0] = 0;
    while (sh.nxt[cur] > cur && sh.nxt[cur] < n && len < a.max_depth) {
      cur = sh.nxt[cur];
      prow[++len] = cur;
      if (cur < 64) w0 |= 1ull << cur;
      else w1 |= 1ull << (cur - 64);
    }
    sh.walked[0] = w0;
    sh.walked[1] = w1;
    sh.tip = cur;
    a.acc_len[b] = len;
    a.bonus[b] = ld_dev(a.ws_sample + n0 + cur);
    sh.len = len;
  }
  wave_lds_sync();
  const int len = sh.len, tip = sh.tip;
  const uint64_t w0 = sh.walked[0], w1 = sh.walked[1];
  for (int s = len + 1 + lane; s <= a.max_depth; s += 64) a.path[(size_t)b * (a.max_depth + 1) + s] = -1;
  int best = kMaxNodes;
  for (int j = lane; j < n; j += 64) {
    const bool walked = j < 64 ? (w0 >> j) & 1 : (w1 >> (j - 64)) & 1;
    uint8_t f = a.flags[n0 + j] & (uint8_t) ~(RESPEC_FLAG_ON_PATH | RESPEC_FLAG_STOCH_ACCEPT);
    if (j > 0 && sh.nxt[sh.par[j]] == j) f |= RESPEC_FLAG_STOCH_ACCEPT;
    if (walked) f |= RESPEC_FLAG_ON_PATH;
    a.flags[n0 + j] = f;
    int la = -1;
    if (!sh.has_child[j]) {
      la = 0;
      bool holds_tip = false;
      for (int v = j, guard = 0; guard <= kMaxDepth; ++guard) {
        const bool wv = v < 64 ? (w0 >> v) & 1 : (w1 >> (v - 64)) & 1;
        la += (v > 0 && wv) ? 1 : 0;
        holds_tip = holds_tip || v == tip;
        if (v == 0) break;
        v = sh.par[v];
      }
      if (holds_tip) best = min(best, j);
    }
    a.leaf_acc_len[n0 + j] = la;
  }
  for (int o = 32; o > 0; o >>= 1) best = min(best, __shfl_xor(best, o, 64));
  if (lane == 0) {
    a.winner_leaf[b] = best < kMaxNodes ? best : -1;
    st_dev(a.seq_counter + b, 0);
  }
}

}  // namespace

hipError_t launch_stochastic(const StochArgs& a, hipStream_t s, hipEvent_t ev_stop) {
  // vocabularies that are a multiple of 4 have 16-byte aligned rows
  if ((a.vocab & 3) == 0)
    return launch_k(stochastic_kernel<true>, dim3(a.total_nodes), dim3(kST), 0, s, nullptr, ev_stop, a);
  return launch_k(stochastic_kernel<false>, dim3(a.total_nodes), dim3(kST), 0, s, nullptr, ev_stop, a);
}

}  // namespace respec
