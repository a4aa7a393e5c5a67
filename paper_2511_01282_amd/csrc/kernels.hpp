// Internal launch interface of the verification kernels (not part of the C ABI).
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace respec {

constexpr int kMaxNodes = 128;   // tree nodes per sequence (ancestor bitsets of 4 words)
constexpr int kMaxDepth = 64;    // chain bits fit one 64-bit mask
constexpr int kVtPad = 4;        // elements of padding per transposed-V row in LDS
constexpr int kKvTile = 32;      // KV rows per wave step in the attention loop

struct AttnArgs {
  const void* hidden;      // [M][Hd]
  const void* k_cache;     // [B][Hkv][kv_cap][D]
  const void* v_cache;
  const int32_t* node_off; // [B+1]
  const int32_t* kv_len;   // [B]
  const int32_t* parent;   // [M]
  float* part_o;           // [B*Hkv*n_rowblk][nsplit][rows_per_wg][D] unnormalised split outputs
  float* part_m;           // [B*Hkv*n_rowblk][nsplit][rows_per_wg]   (log2 units)
  float* part_l;
  void* x_out;             // [M][Hd] residual h + O in the workload dtype (workspace, the LM head's input)
  void* x_copy;            // [M][Hd] the caller's copy of x, or null
  float* attn_out;         // [M][Hd] or null
  int32_t total_nodes, hidden_size, n_kv_heads, group, kv_cap, max_nodes;
  int32_t nsplit, chunk, n_rowblk, rows_per_wg, wr, wk;
  float scale_log2;        // log2(e) / sqrt(D)
  // flat > 0 (register path, 2-64 sequences): blockIdx.x is one of `flat` equal pieces of
  // the KV tiles of every sequence of its head (partial slots per sequence, nsplit = flat);
  // 0: blockIdx.x is a split of `chunk` rows of sequence blockIdx.z
  int32_t flat;
  int32_t batch;
};

struct LmArgs {
  const void* x;           // [M][Hd]
  const void* w;           // [V][Hd]
  float* logits;           // [M][V]
  int32_t m_rows, vocab, hidden_size;
  int32_t n_mtiles;        // tiles of 16*MB token rows
  float* partials;         // [M][n_vtiles][4] per-tile row statistics {m, S, T, argmax}, or null
  int32_t n_vtiles;        // vocabulary tiles of 64 rows
};

struct VocabArgs {
  const float* logits;     // [M][V]
  const float* partials;   // [M][n_vtiles][4] written by the LM-head epilogue
  const int32_t* node_off; // [B+1]
  const int32_t* kv_len;   // [B]
  const int32_t* parent;
  const int32_t* token;
  const uint8_t* src;
  int32_t* seq_counter;    // [B]
  int32_t* flag_ws;        // [M] predicate bits handed from row workgroups to the path reducer
  // outputs
  float* max_logit; float* lse; float* entropy; int32_t* argmax;
  int32_t* topk_id; float* topk_logprob; float* tok_logprob; uint8_t* flags;
  int32_t* leaf_acc_len; int32_t* path; int32_t* acc_len; int32_t* bonus; int32_t* winner_leaf;
  int32_t* seq_status;
  int32_t total_nodes, batch, vocab, n_vtiles, topk_out, max_nodes, max_depth, kv_cap, max_kv;
  int32_t topk, min_lookahead, max_relaxed;
  float tau;
  int32_t stats_only;      // 1: rows write their flags and stop (no ticket, no path reduction)
  int32_t* rank_req;       // [M] workspace: parent row of node i whose rank the rank pass counts, or -1;
                           // null when tok_rank is not requested
  int32_t* tok_rank;       // [M] output, set to 0 (counted by the rank pass) or -1 here; null: not requested
};

struct RankArgs {
  const float* logits;     // [M][V]
  const int32_t* token;    // [M]
  const int32_t* rank_req; // [M] parent row of node j, or -1 (written by the vocabulary pass)
  int32_t* tok_rank;       // [M] zeroed (or -1) by the vocabulary pass; the counts are added here
  int32_t total_nodes, vocab;
};

struct StochArgs {
  const float* logits;     // [M][V]
  const float* max_logit;  // [M] (vocabulary pass)
  const float* lse;        // [M] (vocabulary pass)
  const float* draft_prob; // [M][V] drafter distribution at each node, or null (every draft deterministic)
  const float* uniform;    // [M][2]
  const int32_t* node_off; // [B+1]
  const int32_t* parent;
  const int32_t* token;
  const uint8_t* src;
  const int32_t* seq_status;  // [B] (vocabulary pass)
  int32_t* seq_counter;    // [B], zero between steps
  int32_t* ws_next;        // [M] first accepted child of each node (sequence-local) or -1
  int32_t* ws_sample;      // [M] residual draw of each node or -1
  // outputs
  uint8_t* flags; int32_t* sample; int32_t* leaf_acc_len; int32_t* path; int32_t* acc_len; int32_t* bonus;
  int32_t* winner_leaf;
  int32_t total_nodes, batch, vocab, max_nodes, max_depth;
  float inv_temp;          // 1 / T
  int32_t unit_temp;       // T == 1: the normaliser comes from the log-sum-exp
};

// Launch a kernel whose single argument is an argument struct.  Optional
// start / stop events take the dispatch's own timestamps (hipExtLaunchKernel),
// so a stage timed with them matches the kernel's duration.
template <typename F, typename A>
inline hipError_t launch_k(F kernel, dim3 grid, dim3 block, size_t lds, hipStream_t s, hipEvent_t ev_start,
                           hipEvent_t ev_stop, const A& args) {
  if (ev_start || ev_stop)
    hipExtLaunchKernelGGL(kernel, grid, block, (uint32_t)lds, s, ev_start, ev_stop, 0u, args);
  else
    hipLaunchKernelGGL(kernel, grid, block, lds, s, args);
  return hipGetLastError();
}

// dtype-dispatching launchers (0 = f32, 1 = bf16); return hipSuccess or the launch error.
// ev_start / ev_stop: optional timing events (see launch_k).
hipError_t launch_tree_attn(int dtype, int head_dim, int nb, dim3 grid, int threads, size_t lds,
                            const AttnArgs& a, hipStream_t s, hipEvent_t ev_start = nullptr);
hipError_t set_tree_attn_lds_limit(int dtype, int head_dim, int nb, size_t lds);
hipError_t launch_attn_merge(int dtype, int head_dim, dim3 grid, const AttnArgs& a, hipStream_t s,
                             hipEvent_t ev_stop = nullptr);
// bf16 only; a.wr waves of 32 query rows each (nb = 2) in each of kg (1 or 2)
// key groups, 2-8 waves in all; KV tiles shared through an LDS ring of
// `stages` (8) K+V tiles
hipError_t launch_tree_attn_shared(int head_dim, int nb, int stages, int kg, dim3 grid, int threads, size_t lds,
                                   const AttnArgs& a, hipStream_t s, hipEvent_t ev_start = nullptr);
hipError_t set_tree_attn_shared_lds_limit(int head_dim, int stages, int kg, size_t lds);
constexpr int shared_ring_bytes(int head_dim, int stages) { return stages * 2 * kKvTile * head_dim * 2; }
constexpr int kSharedStages1 = 10;  // ring slots of the shared-tile kernel with one key group (160 KB at head_dim 128)
constexpr int kSharedStages2 = 10;  // ... and with two key groups
// mb: 16-row token blocks per workgroup (1-4 plain, 8 and 16 GEMM); wide: bf16 with up to 64 token
// rows in the GEMM kernel's 256-row vocabulary tiles (n_mtiles = 1)
hipError_t launch_lmhead(int dtype, int mb, bool wide, const LmArgs& a, hipStream_t s, hipEvent_t ev_stop = nullptr);
constexpr int kLmTileRows = 64;  // vocabulary rows per statistics tile (one plain LM-head workgroup)
// Per-tile partial of the vocabulary statistics of one token row over its tile
// of 64 vocabulary rows: {m, S, T, argmax}, 16 bytes.  (m, argmax) is also the
// tile's largest (value, id) key, from which the vocabulary pass bounds the
// row's top-K.
constexpr int kTileWords = 4;
hipError_t launch_finalize(int ko, int blocks, const VocabArgs& a, hipStream_t s, hipEvent_t ev_stop = nullptr);
hipError_t launch_stochastic(const StochArgs& a, hipStream_t s, hipEvent_t ev_stop = nullptr);
// exact ranks of the children's tokens (after the vocabulary pass); chunks of kRankChunk tokens
constexpr int kRankChunk = 4096;
hipError_t launch_rank(const RankArgs& a, hipStream_t s, hipEvent_t ev_stop = nullptr);
constexpr int kMaxStochVocab = 256 * 2048;  // the draw's per-tile masses: 256 tiles of 2048 tokens
hipError_t launch_zero_i32(int32_t* p, size_t n, hipStream_t s);

}  // namespace respec
