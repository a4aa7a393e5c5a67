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
// One workgroup per node row i (after the vocabulary pass, which has written
// the row's max logit and log-sum-exp):
//   - the residual after k rejections is evaluated on the fly from z, the
//     q row and the k normalisers, so a rejection costs one pass over the
//     vocabulary (coalesced 16-byte loads, block-wide sum) and nothing is
//     stored per token;
//   - the children are tested until one passes; if none does, the residual is
//     drawn: each thread sums its contiguous segment of tokens, a block scan
//     gives the segment offsets, and the thread whose segment holds the
//     threshold walks it again;
//   - the row hands its outcome (accepted child, or the draw) to the last row
//     of its sequence (device-scope ticket), which walks the tree from the
//     root along the accepted children and writes the path, the bonus token,
//     the per-leaf accepted lengths and the flags.
#include "../../include/respec_verify.h"
#include "common.hpp"
#include "kernels.hpp"

namespace respec {
namespace {

constexpr int kST = 256;  // threads per row workgroup
constexpr int kSW = kST / 64;

struct StochLds {
  int par[kMaxNodes];
  int tok[kMaxNodes];
  uint8_t src[kMaxNodes];
  int kid[kMaxNodes];       // children of the row (sequence-local), in node order
  int ktok[kMaxNodes];
  uint8_t kmodel[kMaxNodes];
  float kinvz[kMaxNodes];   // 1 / normaliser of each rejected child's residual (0: residual kept)
  uint64_t kids[2];
  float red[kSW];
  float scan[kST];
  int lastpos[kSW];
  int b, n0, n, ok;
  int ticket;
  int sample;
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

// Residual after nrej rejected children, at token v (z: logit, qv: the row's
// draft probability of v or 0).
__device__ __forceinline__ float residual(float z, float qv, int v, int nrej, const StochLds& sh, float m, float inv_t,
                                          float inv_s) {
  float r = __expf((z - m) * inv_t) * inv_s;
  for (int k = 0; k < nrej; ++k) {
    const float iz = sh.kinvz[k];
    if (iz > 0.f) {
      const float q = sh.kmodel[k] ? qv : (v == sh.ktok[k] ? 1.f : 0.f);
      r = fmaxf(r - q, 0.f) * iz;
    }
  }
  return r;
}

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
    const uint64_t m = __ballot(j < n && j > li && sh.par[j] == li);
    if (lane == 0) sh.kids[wave] = m;
  }
  __syncthreads();
  int nk = 0;
  {
    uint64_t m0 = sh.kids[0], m1 = sh.kids[1];
    if (tid == 0) {
      while (m0) {
        const int j = __builtin_ctzll(m0);
        m0 &= m0 - 1;
        sh.ktok[nk] = sh.tok[j];
        sh.kmodel[nk] = a.draft_prob && sh.src[j] != RESPEC_SRC_RETRIEVED;
        sh.kinvz[nk] = 0.f;
        sh.kid[nk] = j;
        ++nk;
      }
      while (m1) {
        const int j = 64 + __builtin_ctzll(m1);
        m1 &= m1 - 1;
        sh.ktok[nk] = sh.tok[j];
        sh.kmodel[nk] = a.draft_prob && sh.src[j] != RESPEC_SRC_RETRIEVED;
        sh.kinvz[nk] = 0.f;
        sh.kid[nk] = j;
        ++nk;
      }
    }
    nk = __popcll(sh.kids[0]) + __popcll(sh.kids[1]);
  }
  __syncthreads();

  const float* zr = a.logits + (size_t)i * a.vocab;
  const float* qr = a.draft_prob ? a.draft_prob + (size_t)i * a.vocab : nullptr;
  const float m = a.max_logit[i];
  const int V = a.vocab;
  const bool vec = (V & 3) == 0;

  // ---- p = softmax(z / T): the normaliser ----
  float inv_s;
  if (a.unit_temp) {
    inv_s = __expf(m - a.lse[i]);
  } else {
    float s = 0.f;
    if (vec) {
      for (int v = 4 * tid; v < V; v += 4 * kST) {
        const f32x4 z4 = *reinterpret_cast<const f32x4*>(zr + v);
        s += __expf((z4.x - m) * a.inv_temp) + __expf((z4.y - m) * a.inv_temp) + __expf((z4.z - m) * a.inv_temp) +
             __expf((z4.w - m) * a.inv_temp);
      }
    } else {
      for (int v = tid; v < V; v += kST) s += __expf((zr[v] - m) * a.inv_temp);
    }
    inv_s = 1.f / block_sum(s, sh, lane, wave);
  }

  // ---- the children, in node order, until one passes ----
  int accepted = -1;
  bool any_model = false;
  for (int k = 0; k < nk; ++k) {
    const int t = sh.ktok[k];
    const bool model = sh.kmodel[k];
    any_model = any_model || model;
    const float qt_row = qr ? qr[t] : 0.f;
    const float rt = residual(zr[t], qt_row, t, k, sh, m, a.inv_temp, inv_s);
    const float qt = model ? qt_row : 1.f;
    const float acc = qt > 0.f ? fminf(rt / qt, 1.f) : (rt > 0.f ? 1.f : 0.f);
    if (a.uniform[2 * (size_t)(n0 + sh.kid[k])] < acc) {
      accepted = k;
      break;
    }
    // rejected: the normaliser of max(r - q_k, 0)
    float s = 0.f;
    const bool rd_q = qr && any_model;
    if (vec) {
      for (int v = 4 * tid; v < V; v += 4 * kST) {
        const f32x4 z4 = *reinterpret_cast<const f32x4*>(zr + v);
        const f32x4 q4 = rd_q ? *reinterpret_cast<const f32x4*>(qr + v) : f32x4{0.f, 0.f, 0.f, 0.f};
        const float zz[4] = {z4.x, z4.y, z4.z, z4.w};
        const float qq[4] = {q4.x, q4.y, q4.z, q4.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float r = residual(zz[e], qq[e], v + e, k, sh, m, a.inv_temp, inv_s);
          const float q = model ? qq[e] : (v + e == t ? 1.f : 0.f);
          s += fmaxf(r - q, 0.f);
        }
      }
    } else {
      for (int v = tid; v < V; v += kST) {
        const float qv = rd_q ? qr[v] : 0.f;
        const float r = residual(zr[v], qv, v, k, sh, m, a.inv_temp, inv_s);
        const float q = model ? qv : (v == t ? 1.f : 0.f);
        s += fmaxf(r - q, 0.f);
      }
    }
    const float z = block_sum(s, sh, lane, wave);
    if (tid == 0) sh.kinvz[k] = z > 0.f ? 1.f / z : 0.f;
    __syncthreads();
  }

  // ---- no child passed: draw from the residual ----
  int sample = -1;
  if (accepted < 0) {
    const bool rd_q = qr && any_model;
    const int seg = (V + kST - 1) / kST;
    const int v0 = tid * seg, v1 = min(V, v0 + seg);
    float part = 0.f;
    int last = -1;
    for (int v = v0; v < v1; ++v) {
      const float r = residual(zr[v], rd_q ? qr[v] : 0.f, v, nk, sh, m, a.inv_temp, inv_s);
      part += r;
      last = r > 0.f ? v : last;
    }
    // block exclusive scan of the segment sums (thread order = token order)
    sh.scan[tid] = part;
    const int lmax = wave_max((float)last);
    if (lane == 0) sh.lastpos[wave] = lmax;
    if (tid == 0) sh.sample = -1;
    __syncthreads();
    float pre = 0.f, total = 0.f;
    for (int u = 0; u < kST; ++u) {
      const float x = sh.scan[u];
      pre += u < tid ? x : 0.f;
      total += x;
    }
    const float thr = a.uniform[2 * (size_t)i + 1] * total;
    if (part > 0.f && pre <= thr && thr < pre + part) {
      float s = 0.f;
      for (int v = v0; v < v1; ++v) {
        s += residual(zr[v], rd_q ? qr[v] : 0.f, v, nk, sh, m, a.inv_temp, inv_s);
        if (pre + s > thr) {
          sh.sample = v;
          break;
        }
      }
    }
    __syncthreads();
    sample = sh.sample;
    if (sample < 0) {  // rounding put the threshold past the last segment: the last token with mass
      int lp = -1;
#pragma unroll
      for (int w = 0; w < kSW; ++w) lp = max(lp, sh.lastpos[w]);
      sample = max(lp, 0);
    }
  }

  // ---- hand-off and the sequence's completion ticket ----
  if (tid == 0) {
    st_dev(a.ws_next + i, accepted >= 0 ? sh.kid[accepted] : -1);
    st_dev(a.ws_sample + i, sample);
    if (a.sample) a.sample[i] = sample;
  }
  stores_done();
  __syncthreads();
  if (tid == 0) sh.ticket = atomicAdd(a.seq_counter + b, 1);
  __syncthreads();
  if (sh.ticket != n - 1 || wave != 0) return;

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
  return launch_k(stochastic_kernel, dim3(a.total_nodes), dim3(kST), 0, s, nullptr, ev_stop, a);
}

}  // namespace respec
