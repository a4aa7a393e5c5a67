// Host side of the respec_verify C ABI: plan creation (tiling choices and
// workspace layout), argument validation and the launch sequence of one
// verification step.  See include/respec_verify.h for the contract.
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <atomic>
#include <mutex>
#include <new>

#include "../../include/respec_verify.h"
#include "kernels.hpp"

using namespace respec;

struct respec_verify_plan {
  respec_verify_shape s;
  int es;                 // bytes per element of the workload dtype
  int group;              // Hq / Hkv
  // attention tiling
  int nb, wr, wk, rows_per_wg, n_rowblk, attn_threads, nsplit_cap;
  int attn_shared;        // bf16 with several waves of rows per KV head: KV tiles shared through LDS
  int attn_stages;        // ring slots of the shared-tile kernel
  int attn_kg;            // key groups of the shared-tile kernel
  int attn_wg_target;     // workgroups the splits aim for
  int flat_pieces;        // ragged batches (register path): pieces of each head's KV tiles
  size_t attn_lds;
  // vocabulary statistics: tiles of the LM head and the top-K width (8 or 16)
  int ko, n_vtiles;
  // workspace layout (bytes)
  size_t off_po, off_pm, off_pl, off_x, off_part, off_flag, off_cnt, off_stoch, off_rank;
  size_t n_cnt_seq, total;
  // the attention kernel's LDS limit is raised on the first step (plan creation stays GPU-free)
  mutable std::atomic<bool> lds_ready{false};
};

namespace {

constexpr int kTargetWaves = 1024;  // attention: one wave per SIMD on a 256-CU MI355X
constexpr int kCUs = 256;

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
int cdiv(long long a, long long b) { return (int)((a + b - 1) / b); }
int clampi(int x, int lo, int hi) { return x < lo ? lo : (x > hi ? hi : x); }
bool aligned(const void* p, size_t n) { return ((uintptr_t)p % n) == 0; }

}  // namespace

extern "C" {

const char* respec_status_string(respec_status st) {
  switch (st) {
    case RESPEC_OK: return "ok";
    case RESPEC_ERR_NULL: return "a required pointer is NULL";
    case RESPEC_ERR_SHAPE: return "sizes out of the supported range or inconsistent";
    case RESPEC_ERR_DTYPE: return "unknown dtype";
    case RESPEC_ERR_PARAM: return "acceptance parameters out of range";
    case RESPEC_ERR_TREE: return "malformed draft tree";
    case RESPEC_ERR_CAPACITY: return "batch, nodes or KV length above the plan's capacity";
    case RESPEC_ERR_HIP: return "HIP call or kernel launch failed";
    case RESPEC_ERR_WORKSPACE: return "workspace missing or not 256-byte aligned";
    case RESPEC_ERR_TOKEN: return "draft token or source tag out of range";
    case RESPEC_ERR_SCRATCH: return "plan needs more workspace or sequences than the static scratch of the allocation-free step holds";
  }
  return "unknown status";
}

respec_status respec_verify_check_tree(const int32_t* parent, int32_t n, int32_t max_depth) {
  if (!parent) return RESPEC_ERR_NULL;
  if (n < 1 || n > RESPEC_MAX_NODES || max_depth < 0) return RESPEC_ERR_SHAPE;
  if (parent[0] != -1) return RESPEC_ERR_TREE;
  int depth[RESPEC_MAX_NODES];
  depth[0] = 0;
  for (int j = 1; j < n; ++j) {
    if (parent[j] < 0 || parent[j] >= j) return RESPEC_ERR_TREE;
    depth[j] = depth[parent[j]] + 1;
    if (depth[j] > max_depth) return RESPEC_ERR_TREE;
  }
  return RESPEC_OK;
}

respec_status respec_verify_create(const respec_verify_shape* shape, respec_verify_plan** out) {
  if (!shape || !out) return RESPEC_ERR_NULL;
  *out = nullptr;
  const respec_verify_shape& s = *shape;
  if (s.dtype != RESPEC_F32 && s.dtype != RESPEC_BF16) return RESPEC_ERR_DTYPE;
  if (s.head_dim != 64 && s.head_dim != 128) return RESPEC_ERR_SHAPE;
  if (s.n_q_heads < 1 || s.n_kv_heads < 1 || s.n_q_heads % s.n_kv_heads != 0) return RESPEC_ERR_SHAPE;
  if ((long long)s.n_q_heads * s.head_dim != s.hidden) return RESPEC_ERR_SHAPE;
  const int es = s.dtype == RESPEC_BF16 ? 2 : 4;
  if (((long long)s.hidden * es) % 512 != 0) return RESPEC_ERR_SHAPE;
  if (s.topk_out < 1 || s.topk_out > RESPEC_MAX_TOPK_OUT || s.vocab < s.topk_out) return RESPEC_ERR_SHAPE;
  if (s.max_batch < 1 || s.max_nodes < 1 || s.max_nodes > RESPEC_MAX_NODES) return RESPEC_ERR_SHAPE;
  if (s.max_depth < 0 || s.max_depth > RESPEC_MAX_DEPTH || s.max_kv_len < 0) return RESPEC_ERR_SHAPE;
  if ((long long)s.max_batch * s.max_nodes > (1ll << 24)) return RESPEC_ERR_SHAPE;

  respec_verify_plan* p = new (std::nothrow) respec_verify_plan();
  if (!p) return RESPEC_ERR_SHAPE;
  p->s = s;
  p->es = es;
  p->group = s.n_q_heads / s.n_kv_heads;

  // attention: rows of a KV head are (node, head-in-group) pairs; a wave owns
  // at most 32 of them (more would not fit the registers next to a ring of
  // tiles); above 4 waves' worth a head's KV rows are read once per row block
  const int rmax = s.max_nodes * p->group;
  const int nb = rmax <= 16 ? 1 : 2;
  const int rg = cdiv(rmax, 16 * nb);
  const int rb = 16 * nb;
  const long long t_cap = (long long)s.max_kv_len + s.max_nodes;
  p->nb = nb;
  p->attn_shared = es == 2 && rg >= 2;
  if (p->attn_shared) {
    // up to 8 waves of rows read every KV tile once, from a shared LDS ring,
    // one workgroup per CU; up to 4 waves of rows, a second key group of as
    // many waves takes every other tile (one workgroup fills the CU, and its
    // two halves stay in step)
    p->wr = rg < 8 ? rg : 8;
    p->n_rowblk = cdiv(rg, p->wr);
    p->wk = 1;
    p->attn_kg = p->wr <= 4 ? 2 : 1;
    p->rows_per_wg = p->wr * rb;
    p->attn_threads = 64 * p->wr * p->attn_kg;
    p->attn_stages = p->attn_kg == 1 ? kSharedStages1 : kSharedStages2;
    p->attn_lds = (size_t)shared_ring_bytes(s.head_dim, p->attn_stages);
    p->attn_wg_target = kCUs;
  } else {
    p->wr = rg < 4 ? rg : 4;
    p->n_rowblk = cdiv(rg, p->wr);
    int wk = 4 / p->wr;
    if (wk > 128 / (p->wr * rb)) wk = 128 / (p->wr * rb);
    p->wk = wk < 1 ? 1 : wk;
    p->rows_per_wg = p->wr * rb;
    const int nwaves = p->wr * p->wk;
    p->attn_threads = 64 * nwaves;
    // per wave: one row-major, swizzled V tile (bf16) or one transposed, padded V tile (float32)
    const size_t vt_bytes = es == 2 ? (size_t)nwaves * kKvTile * s.head_dim * es
                                    : (size_t)nwaves * s.head_dim * (kKvTile + kVtPad) * es;
    // wave merge: every wave's O lane-major (D/16 x NB blocks of 64 x 16 bytes) plus its m and l
    const size_t merge_bytes =
        p->wk > 1 ? (size_t)nwaves * ((size_t)(s.head_dim / 16) * p->nb * 64 * 16 + (size_t)2 * p->nb * 64 * 4) : 0;
    p->attn_lds = vt_bytes > merge_bytes ? vt_bytes : merge_bytes;
    p->attn_wg_target = kTargetWaves / nwaves;
  }
  const int per_split = s.n_kv_heads * p->n_rowblk;
  p->nsplit_cap = clampi(p->attn_wg_target / per_split, 1, cdiv(t_cap, kKvTile));
  // one piece per CU (two per CU measured slower on an 8-sequence ragged batch: 158 against 144 us)
  p->flat_pieces = p->attn_shared ? 0 : clampi(p->attn_wg_target / per_split, 1, 64);
  const int slots = p->nsplit_cap > p->flat_pieces ? p->nsplit_cap : p->flat_pieces;

  p->ko = s.topk_out <= 8 ? 8 : 16;
  p->n_vtiles = cdiv(s.vocab, kLmTileRows);

  // workspace
  const size_t mcap = (size_t)s.max_batch * s.max_nodes;
  const size_t prow = (size_t)s.max_batch * s.n_kv_heads * p->n_rowblk * slots * p->rows_per_wg;
  size_t off = 0;
  p->off_po = off; off = align256(off + prow * s.head_dim * 4);
  p->off_pm = off; off = align256(off + prow * 4);
  p->off_pl = off; off = align256(off + prow * 4);
  p->off_x = off; off = align256(off + mcap * s.hidden * es);
  p->off_part = off; off = align256(off + mcap * p->n_vtiles * kTileWords * 4);
  p->off_flag = off; off = align256(off + mcap * 4);
  p->n_cnt_seq = s.max_batch;
  p->off_cnt = off; off = align256(off + p->n_cnt_seq * 4);
  p->off_stoch = off; off = align256(off + 2 * mcap * 4);  // stochastic walk: next child, draw
  p->off_rank = off; off = align256(off + mcap * 4);       // rank requests: parent row per node
  p->total = off;

  *out = p;
  return RESPEC_OK;
}

void respec_verify_destroy(respec_verify_plan* plan) { delete plan; }

size_t respec_verify_workspace_bytes(const respec_verify_plan* plan) { return plan ? plan->total : 0; }

respec_status respec_verify_workspace_init(const respec_verify_plan* plan, void* workspace, void* stream) {
  if (!plan) return RESPEC_ERR_NULL;
  if (!workspace || !aligned(workspace, 256)) return RESPEC_ERR_WORKSPACE;
  int32_t* cnt = reinterpret_cast<int32_t*>(static_cast<char*>(workspace) + plan->off_cnt);
  const size_t n = plan->n_cnt_seq;
  return launch_zero_i32(cnt, n, static_cast<hipStream_t>(stream)) == hipSuccess ? RESPEC_OK : RESPEC_ERR_HIP;
}

}  // extern "C"

namespace {

// One step on workspace `ws` (the plan's layout) with the sequences' completion
// counters at `cnt` (zero between steps).
respec_status step_impl(const respec_verify_plan* plan, const respec_verify_args* args, char* ws, int32_t* cnt,
                        void* stream) {
  const respec_verify_shape& s = plan->s;
  const respec_verify_args& a = *args;
  if (a.stop_after < RESPEC_STOP_ALL || a.stop_after > RESPEC_STOP_STATS) return RESPEC_ERR_PARAM;
  if (a.batch < 0) return RESPEC_ERR_SHAPE;
  if (a.batch > s.max_batch) return RESPEC_ERR_CAPACITY;
  const bool full = a.stop_after == RESPEC_STOP_ALL;
  const bool stats_only = a.stop_after == RESPEC_STOP_STATS;
  const bool vocab_pass = full || stats_only;  // statistics and predicates run
  const bool need_logits = a.stop_after != RESPEC_STOP_ATTN;
  if (vocab_pass) {
    const respec_accept_params& q = a.accept;
    if (q.topk < 1 || q.topk > s.topk_out || !(q.tau >= 0.f) || isinf(q.tau) || q.min_lookahead < 0 ||
        q.max_relaxed < 0 || (q.stochastic != 0 && q.stochastic != 1))
      return RESPEC_ERR_PARAM;
    if (q.stochastic && (!(q.temperature > 0.f) || isinf(q.temperature))) return RESPEC_ERR_PARAM;
    if (q.stochastic && s.vocab > kMaxStochVocab) return RESPEC_ERR_SHAPE;
  }
  const bool stochastic = full && a.accept.stochastic;
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipEvent_t* ev = static_cast<hipEvent_t*>(a.stage_events);
  if (a.batch == 0) {
    if (ev)
      for (int k = 0; k < 4; ++k)
        if (hipEventRecord(ev[k], st) != hipSuccess) return RESPEC_ERR_HIP;
    return RESPEC_OK;
  }
  if (a.max_nodes_in_batch < 1 || a.max_kv_len_in_batch < 0) return RESPEC_ERR_SHAPE;
  if (a.max_nodes_in_batch > s.max_nodes || a.max_kv_len_in_batch > s.max_kv_len) return RESPEC_ERR_CAPACITY;
  if (a.total_nodes < a.batch || (long long)a.total_nodes > (long long)a.batch * a.max_nodes_in_batch)
    return RESPEC_ERR_SHAPE;
  if ((long long)a.kv_capacity < (long long)a.max_kv_len_in_batch + a.max_nodes_in_batch) return RESPEC_ERR_SHAPE;
  if (!a.node_off || !a.kv_len || !a.hidden || !a.k_cache || !a.v_cache || !a.parent) return RESPEC_ERR_NULL;
  if (need_logits && (!a.lm_head || !a.logits)) return RESPEC_ERR_NULL;
  if (vocab_pass && (!a.token || !a.src || !a.max_logit || !a.lse || !a.entropy || !a.argmax || !a.topk_id ||
                     !a.topk_logprob || !a.tok_logprob || !a.flags))
    return RESPEC_ERR_NULL;
  if (full && (!a.leaf_acc_len || !a.path || !a.acc_len || !a.bonus || !a.winner_leaf || !a.seq_status))
    return RESPEC_ERR_NULL;
  if (stochastic && !a.uniform) return RESPEC_ERR_NULL;
  if (stochastic && a.draft_prob && !aligned(a.draft_prob, 16)) return RESPEC_ERR_SHAPE;
  if (!aligned(a.hidden, 16) || !aligned(a.k_cache, 16) || !aligned(a.v_cache, 16) ||
      (need_logits && (!aligned(a.lm_head, 16) || !aligned(a.logits, 16))) || (a.attn_out && !aligned(a.attn_out, 16)))
    return RESPEC_ERR_SHAPE;
  const bool rank = vocab_pass && a.tok_rank != nullptr;


  if (!plan->lds_ready.load(std::memory_order_acquire)) {
    const hipError_t e = plan->attn_shared ? set_tree_attn_shared_lds_limit(s.head_dim, plan->attn_stages, plan->attn_kg, plan->attn_lds)
                                           : set_tree_attn_lds_limit(s.dtype, s.head_dim, plan->nb, plan->attn_lds);
    if (e != hipSuccess) return RESPEC_ERR_HIP;
    plan->lds_ready.store(true, std::memory_order_release);
  }

  // ---- tree-masked attention + residual ----
  AttnArgs at;
  at.hidden = a.hidden;
  at.k_cache = a.k_cache;
  at.v_cache = a.v_cache;
  at.node_off = a.node_off;
  at.kv_len = a.kv_len;
  at.parent = a.parent;
  at.part_o = reinterpret_cast<float*>(ws + plan->off_po);
  at.part_m = reinterpret_cast<float*>(ws + plan->off_pm);
  at.part_l = reinterpret_cast<float*>(ws + plan->off_pl);
  at.x_out = ws + plan->off_x;
  at.attn_out = a.attn_out;
  at.x_copy = a.x_out;
  at.total_nodes = a.total_nodes;
  at.hidden_size = s.hidden;
  at.n_kv_heads = s.n_kv_heads;
  at.group = plan->group;
  at.kv_cap = a.kv_capacity;
  at.max_nodes = a.max_nodes_in_batch;
  const long long t_max = (long long)a.max_kv_len_in_batch + a.max_nodes_in_batch;
  const int per_split = a.batch * s.n_kv_heads * plan->n_rowblk;
  const int target = clampi(plan->attn_wg_target / per_split, 1, plan->nsplit_cap);
  // (a split holds at least one tile per key-group wave: fewer, fuller splits for short caches)
  at.chunk = max(cdiv(cdiv(t_max, target), kKvTile), plan->attn_shared ? plan->attn_kg : plan->wk) * kKvTile;
  at.nsplit = cdiv(t_max, at.chunk);
  at.flat = 0;
  at.batch = a.batch;
  // Ragged batches on the register path: each head's KV tiles over every sequence are cut
  // into equal pieces, one workgroup each, so that the longest sequence does not finish
  // alone (per-sequence splits leave every other workgroup idle at the end).
  const bool flat = !plan->attn_shared && a.batch > 1 && a.batch <= 64;
  if (flat) {
    at.flat = plan->flat_pieces;
    at.nsplit = at.flat;
    at.chunk = 0;
  }
  at.n_rowblk = plan->n_rowblk;
  at.rows_per_wg = plan->rows_per_wg;
  at.wr = plan->wr;
  at.wk = plan->wk;
  at.scale_log2 = (float)(1.4426950408889634 / sqrt((double)s.head_dim));
  dim3 agrid(at.nsplit, s.n_kv_heads * plan->n_rowblk, flat ? 1 : a.batch);
  hipError_t ae;
  if (plan->attn_shared)
    ae = launch_tree_attn_shared(s.head_dim, plan->nb, plan->attn_stages, plan->attn_kg, agrid, plan->attn_threads,
                                 plan->attn_lds, at, st, ev ? ev[0] : nullptr);
  else
    ae = launch_tree_attn(s.dtype, s.head_dim, plan->nb, agrid, plan->attn_threads, plan->attn_lds, at, st,
                          ev ? ev[0] : nullptr);
  if (ae != hipSuccess) return RESPEC_ERR_HIP;
  const int merge_rows = 256 / (s.head_dim / 4);
  dim3 mgrid(cdiv(plan->rows_per_wg, merge_rows), a.batch * s.n_kv_heads * plan->n_rowblk);
  if (launch_attn_merge(s.dtype, s.head_dim, mgrid, at, st, ev ? ev[1] : nullptr) != hipSuccess)
    return RESPEC_ERR_HIP;

  // ---- LM head ----
  if (need_logits) {
    LmArgs lm;
    lm.x = ws + plan->off_x;
    lm.w = a.lm_head;
    lm.logits = a.logits;
    lm.m_rows = a.total_nodes;
    lm.vocab = s.vocab;
    lm.hidden_size = s.hidden;
    // token rows per workgroup 16*mb: up to 64 in the plain kernel, 128 or 256
    // in the GEMM one (bf16), so that W is streamed once for up to 256 rows.  A vocabulary of more 64-row tiles than two per CU takes
    // the GEMM kernel's 256-row vocabulary tiles (bf16): each x row then serves
    // four times as many W rows.
    const int M = a.total_nodes;
    int mb = M <= 16 ? 1 : M <= 32 ? 2 : M <= 48 ? 3 : 4;
    if (M > 64 && s.dtype == RESPEC_BF16) mb = M <= 128 ? 8 : 16;
    const bool wide = s.dtype == RESPEC_BF16 && M <= 64 && plan->n_vtiles > 2 * kCUs;
    lm.n_mtiles = wide ? 1 : cdiv(M, 16 * mb);
    lm.partials = vocab_pass ? reinterpret_cast<float*>(ws + plan->off_part) : nullptr;
    lm.n_vtiles = plan->n_vtiles;
    if (launch_lmhead(s.dtype, mb, wide, lm, st, ev ? ev[2] : nullptr) != hipSuccess) return RESPEC_ERR_HIP;
  } else if (ev && hipEventRecord(ev[2], st) != hipSuccess) {
    return RESPEC_ERR_HIP;
  }

  // ---- row statistics, predicates, path ----
  if (vocab_pass) {
    VocabArgs v;
    v.logits = a.logits;
    v.partials = reinterpret_cast<const float*>(ws + plan->off_part);
    v.node_off = a.node_off;
    v.kv_len = a.kv_len;
    v.parent = a.parent;
    v.token = a.token;
    v.src = a.src;
    v.seq_counter = cnt;
    v.flag_ws = reinterpret_cast<int32_t*>(ws + plan->off_flag);
    v.max_logit = a.max_logit;
    v.lse = a.lse;
    v.entropy = a.entropy;
    v.argmax = a.argmax;
    v.topk_id = a.topk_id;
    v.topk_logprob = a.topk_logprob;
    v.tok_logprob = a.tok_logprob;
    v.flags = a.flags;
    v.leaf_acc_len = a.leaf_acc_len;
    v.path = a.path;
    v.acc_len = a.acc_len;
    v.bonus = a.bonus;
    v.winner_leaf = a.winner_leaf;
    v.seq_status = a.seq_status;
    v.total_nodes = a.total_nodes;
    v.batch = a.batch;
    v.vocab = s.vocab;
    v.n_vtiles = plan->n_vtiles;
    v.topk_out = s.topk_out;
    v.max_nodes = a.max_nodes_in_batch;
    v.max_depth = s.max_depth;
    v.kv_cap = a.kv_capacity;
    v.max_kv = a.max_kv_len_in_batch;
    v.topk = a.accept.topk;
    v.min_lookahead = a.accept.min_lookahead;
    v.max_relaxed = a.accept.max_relaxed;
    v.tau = a.accept.tau;
    v.stats_only = stats_only;
    v.rank_req = rank ? reinterpret_cast<int32_t*>(ws + plan->off_rank) : nullptr;
    v.tok_rank = rank ? a.tok_rank : nullptr;
    // (the stage's last kernel takes the stop event: the rank pass, else the sampling walk, else this one)
    if (launch_finalize(plan->ko, a.total_nodes + a.batch, v, st, (ev && !stochastic && !rank) ? ev[3] : nullptr) !=
        hipSuccess)
      return RESPEC_ERR_HIP;
    if (stochastic) {
      // speculative-sampling walk, after the row statistics and the tree checks
      StochArgs sa;
      sa.logits = a.logits;
      sa.max_logit = a.max_logit;
      sa.lse = a.lse;
      sa.draft_prob = a.draft_prob;
      sa.uniform = a.uniform;
      sa.node_off = a.node_off;
      sa.parent = a.parent;
      sa.token = a.token;
      sa.src = a.src;
      sa.seq_status = a.seq_status;
      sa.seq_counter = cnt;
      sa.ws_next = reinterpret_cast<int32_t*>(ws + plan->off_stoch);
      sa.ws_sample = sa.ws_next + (size_t)s.max_batch * s.max_nodes;
      sa.flags = a.flags;
      sa.sample = a.sample;
      sa.leaf_acc_len = a.leaf_acc_len;
      sa.path = a.path;
      sa.acc_len = a.acc_len;
      sa.bonus = a.bonus;
      sa.winner_leaf = a.winner_leaf;
      sa.total_nodes = a.total_nodes;
      sa.batch = a.batch;
      sa.vocab = s.vocab;
      sa.max_nodes = a.max_nodes_in_batch;
      sa.max_depth = s.max_depth;
      sa.inv_temp = 1.f / a.accept.temperature;
      sa.unit_temp = a.accept.temperature == 1.f;
      if (launch_stochastic(sa, st, (ev && !rank) ? ev[3] : nullptr) != hipSuccess) return RESPEC_ERR_HIP;
    }
    if (rank) {
      RankArgs ra;
      ra.logits = a.logits;
      ra.token = a.token;
      ra.rank_req = v.rank_req;
      ra.tok_rank = a.tok_rank;
      ra.total_nodes = a.total_nodes;
      ra.vocab = s.vocab;
      if (launch_rank(ra, st, ev ? ev[3] : nullptr) != hipSuccess) return RESPEC_ERR_HIP;
    }
  } else if (ev && hipEventRecord(ev[3], st) != hipSuccess) {
    return RESPEC_ERR_HIP;
  }
  return RESPEC_OK;
}

// ---- static workspace of the allocation-free entry point ----
// The array's name is a host-side stand-in: host code uses the device address
// that hipGetSymbolAddress returns for the current device, never `scratch`.
// The front kScratchCounterBytes hold the completion counters at a fixed place,
// so that plans with different workspace layouts sharing the array never read
// another plan's leftovers as counters; the plan's workspace follows them.
constexpr size_t kScratchBytes = (size_t)RESPEC_NOALLOC_SCRATCH_BYTES;
constexpr size_t kScratchCounterBytes = (size_t)RESPEC_NOALLOC_MAX_BATCH * 4;
static_assert(kScratchCounterBytes % 256 == 0, "the workspace after the counters stays 256-byte aligned");
constexpr int kMaxDevices = 64;

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

struct ScratchSlot {
  std::once_flag once;
  char* ptr = nullptr;  // device address of `scratch` on this device (null: set-up failed)
};
ScratchSlot g_scratch[kMaxDevices];

// Device address of this device's array; on the first call on a device (with
// that device current) it is looked up and the counters are cleared by a fill
// kernel on `stream` (no memset node, so a captured first call stays correct).
char* scratch_for_current_device(hipStream_t stream) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  ScratchSlot& sl = g_scratch[dev];
  std::call_once(sl.once, [&] {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return;
    if (launch_zero_i32(static_cast<int32_t*>(p), RESPEC_NOALLOC_MAX_BATCH, stream) != hipSuccess) return;
    sl.ptr = static_cast<char*>(p);
  });
  return sl.ptr;
}

}  // namespace

extern "C" {

respec_status respec_verify_step(const respec_verify_plan* plan, const respec_verify_args* args, void* workspace,
                                 void* stream) {
  if (!plan || !args) return RESPEC_ERR_NULL;
  if (!workspace || !aligned(workspace, 256)) return RESPEC_ERR_WORKSPACE;
  char* ws = static_cast<char*>(workspace);
  return step_impl(plan, args, ws, reinterpret_cast<int32_t*>(ws + plan->off_cnt), stream);
}

respec_status respec_verify_step_noalloc(const respec_verify_plan* plan, const respec_verify_args* args,
                                         void* stream) {
  if (!plan || !args) return RESPEC_ERR_NULL;
  if (plan->total > kScratchBytes - kScratchCounterBytes || plan->s.max_batch > RESPEC_NOALLOC_MAX_BATCH)
    return RESPEC_ERR_SCRATCH;
  char* base = scratch_for_current_device(static_cast<hipStream_t>(stream));
  if (!base) return RESPEC_ERR_HIP;
  return step_impl(plan, args, base + kScratchCounterBytes, reinterpret_cast<int32_t*>(base), stream);
}

}  // extern "C"
