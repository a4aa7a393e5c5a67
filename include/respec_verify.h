/* respec_verify.h -- C ABI for one draft-tree verification step on MI355X (gfx950).
 *
 * The operation is the verification core of retrieval-enhanced speculative
 * decoding (ReSpec, arXiv 2511.01282): a target model checks, in one parallel
 * pass, a draft tree that merges retrieved and model-drafted candidates
 * (Section 3.5, Algorithm 1: BuildDraftTree, RelaxedVerify / StrictVerify).
 * Each draft token carries its source; model drafts are verified strictly
 * (greedy), retrieved drafts with the relaxed check of Eq. 6-7 and the
 * look-ahead tolerance procedure (Section 3.4).  The step also returns the
 * per-node Shannon entropy of the target distribution (Eq. 1, the signal of
 * the entropy-guided trigger, Section 3.2.1) and the per-candidate accepted
 * lengths that feed the EMA score update (Eq. 4-5, Section 3.3).
 *
 * The target forward is a one-layer proxy: for node i the query of head h is
 * the node's hidden state viewed as heads, q = hidden[i][h*D .. h*D+D); it
 * attends (scale 1/sqrt(D)) to every prefix row of its sequence's KV cache and
 * to the tree rows of its ancestors and itself (tree mask); x = round(h + O)
 * in the workload dtype feeds the LM head z = x W^T; p = softmax(z).
 *
 * Conventions
 *  - Every tensor pointer in respec_verify_args is caller-owned DEVICE memory.
 *    Functions marked "host" take host pointers.  hidden, k_cache, v_cache,
 *    lm_head, logits and attn_out must be 16-byte aligned (RESPEC_ERR_SHAPE).
 *  - The library never allocates, frees or synchronises device memory; a step
 *    only enqueues kernels on the caller's stream (a hipStream_t passed as
 *    void*, NULL = the null stream).  It can be captured in a hipGraph.
 *  - A plan holds host metadata only and is immutable after creation; it may be
 *    shared by threads.  Each stream that runs steps concurrently needs its own
 *    workspace.
 *  - Host-side argument checks return a status and launch nothing.  Errors in
 *    device data (malformed parent arrays, out-of-range tokens or tags, bad
 *    node offsets) are reported per sequence in seq_status[b]; the kernels
 *    never trap and never read outside the buffers described here.
 *  - No exceptions cross this ABI and nothing is printed.
 */
#ifndef RESPEC_VERIFY_H
#define RESPEC_VERIFY_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  RESPEC_OK = 0,
  RESPEC_ERR_NULL = 1,      /* a required pointer is NULL                                  */
  RESPEC_ERR_SHAPE = 2,     /* sizes out of the supported range or inconsistent             */
  RESPEC_ERR_DTYPE = 3,     /* unknown dtype                                                */
  RESPEC_ERR_PARAM = 4,     /* acceptance parameters out of range                           */
  RESPEC_ERR_TREE = 5,      /* malformed draft tree (host check, or seq_status on device)   */
  RESPEC_ERR_CAPACITY = 6,  /* batch / nodes / KV length above the plan's capacity          */
  RESPEC_ERR_HIP = 7,       /* a HIP call or kernel launch failed                            */
  RESPEC_ERR_WORKSPACE = 8, /* workspace missing or not 256-byte aligned                    */
  RESPEC_ERR_TOKEN = 9,     /* seq_status only: a draft token or source tag is out of range */
  RESPEC_ERR_SCRATCH = 10   /* respec_verify_step_noalloc: the plan does not fit the static scratch */
} respec_status;

typedef enum { RESPEC_F32 = 0, RESPEC_BF16 = 1 } respec_dtype;

/* Source tag of a draft node (Section 3.4: source-aware verification).
 * The root's tag is ignored. */
typedef enum { RESPEC_SRC_MODEL = 0, RESPEC_SRC_RETRIEVED = 1 } respec_src;

/* flags[j] bits, describing node j's own draft token t_j against the target
 * distribution p_i of its parent i. */
enum {
  RESPEC_FLAG_GREEDY = 1,   /* t_j == argmax p_i (strict, greedy verification)            */
  RESPEC_FLAG_TOPK = 2,     /* t_j in TopK_k(p_i), ties by smaller token id (Eq. 6)         */
  RESPEC_FLAG_TAU = 4,      /* log p_i(argmax) - log p_i(t_j) <= tau (Eq. 7)                */
  RESPEC_FLAG_RELAXED = 8,  /* src_j == RETRIEVED and TOPK and TAU                          */
  RESPEC_FLAG_ON_PATH = 16, /* node is on the accepted path (the root always is)            */
  RESPEC_FLAG_STOCH_ACCEPT = 32 /* stochastic mode: the first child of its parent that passes
                                   the speculative-sampling test (see respec_accept_params)   */
};

/* stop_after (debugging and per-stage timing).  ATTN: attention and residual
 * only (attn_out, x_out); LOGITS: also the LM head (logits); STATS: also the
 * per-row statistics and per-node predicates (max_logit, lse, entropy, argmax,
 * topk_id, topk_logprob, tok_logprob, tok_rank, flags without ON_PATH), but no
 * path reduction (leaf_acc_len, path, acc_len, bonus, winner_leaf, seq_status
 * and sample are not written and may be NULL); ALL: the whole step. */
enum { RESPEC_STOP_ALL = 0, RESPEC_STOP_ATTN = 1, RESPEC_STOP_LOGITS = 2, RESPEC_STOP_STATS = 3 };

/* Limits of this implementation. */
enum { RESPEC_MAX_NODES = 128, RESPEC_MAX_DEPTH = 64, RESPEC_MAX_TOPK_OUT = 16 };

/* Static scratch of respec_verify_step_noalloc: 64 MiB of device memory per GPU
 * (the front 64 KiB hold one completion counter per sequence, the rest the
 * plan's workspace), so plans with respec_verify_workspace_bytes() up to
 * RESPEC_NOALLOC_SCRATCH_BYTES - 4 * RESPEC_NOALLOC_MAX_BATCH and max_batch up
 * to RESPEC_NOALLOC_MAX_BATCH. */
#define RESPEC_NOALLOC_SCRATCH_BYTES (64u << 20)
#define RESPEC_NOALLOC_MAX_BATCH 16384

/* Shapes and capacities, fixed when the plan is created. */
typedef struct {
  int32_t hidden;      /* Hd = n_q_heads * head_dim                                       */
  int32_t n_q_heads;   /* Hq                                                               */
  int32_t n_kv_heads;  /* Hkv, divides Hq (grouped-query attention)                        */
  int32_t head_dim;    /* D: 64 or 128                                                     */
  int32_t vocab;       /* V >= topk_out                                                    */
  int32_t dtype;       /* respec_dtype of hidden, K/V cache and LM head                    */
  int32_t max_batch;   /* capacity in sequences                                            */
  int32_t max_nodes;   /* capacity in tree nodes per sequence, <= RESPEC_MAX_NODES         */
  int32_t max_depth;   /* capacity in tree depth (edges), <= RESPEC_MAX_DEPTH              */
  int32_t max_kv_len;  /* capacity in prefix length per sequence                           */
  int32_t topk_out;    /* width of the top-k output, 1..RESPEC_MAX_TOPK_OUT                */
} respec_verify_shape;

/* Acceptance parameters (Section 3.4), per call.
 *
 * stochastic = 0 (the paper's experiments): model-drafted nodes are verified
 * strictly and greedily (token == argmax), retrieved nodes with the relaxed
 * check and the look-ahead tolerance procedure; the longest accepted chain wins.
 *
 * stochastic = 1: lossless speculative sampling (Section 3.4, drafter outputs)
 * at temperature T, p = softmax(z / T).  A node tries its children in node
 * order; child j passes with probability min(1, r(t_j) / q_j(t_j)), decided by
 * uniform[j][0] < that probability, where r is the node's p with the residual
 * of every earlier rejected sibling k applied, r <- norm(max(r - q_k, 0)) (kept
 * as it is when that has no mass).  q_j is row i of draft_prob for a MODEL
 * child of node i and one-hot at t_j for a RETRIEVED child (a deterministic
 * draft; also for every child when draft_prob is NULL).  The walk starts at the
 * root and moves to the first passing child until none passes; path, acc_len
 * and ON_PATH describe it, bonus is the residual draw at its last node (the
 * smallest token whose cumulative residual mass exceeds uniform[i][1] times
 * the total), winner_leaf the smallest leaf below that node, leaf_acc_len the
 * walked nodes on each leaf's chain.  GREEDY/TOPK/TAU/RELAXED are still
 * reported (at T = 1), and so are the statistics. */
typedef struct {
  int32_t topk;          /* k of TopK_k, 1 <= k <= topk_out                               */
  float tau;             /* tolerance margin, >= 0 (in nats = logit units)                 */
  int32_t min_lookahead; /* m: greedy matches required after a relaxed token, >= 0         */
  int32_t max_relaxed;   /* Phi: relaxed attempts per candidate chain, >= 0                */
  int32_t stochastic;    /* 0: greedy strict / relaxed verification; 1: speculative sampling
                            (vocab <= 524288, else RESPEC_ERR_SHAPE)                    */
  float temperature;     /* T of stochastic verification, finite and > 0                   */
} respec_accept_params;

typedef struct {
  /* host scalars */
  int32_t batch;               /* B, 0 <= B <= max_batch                                  */
  int32_t total_nodes;         /* M = node_off[B]; rows of the per-node tensors            */
  int32_t max_nodes_in_batch;  /* >= every node_off[b+1]-node_off[b], <= max_nodes        */
  int32_t max_kv_len_in_batch; /* >= every kv_len[b], <= max_kv_len                       */
  int32_t kv_capacity;         /* L_cap, rows per head in the cache, >= max_kv_len_in_batch
                                  + max_nodes_in_batch                                     */
  int32_t stop_after;          /* RESPEC_STOP_*                                            */
  respec_accept_params accept;

  /* inputs (device) */
  const int32_t* node_off;  /* [B+1] int32, node_off[0] = 0: sequence b owns global nodes
                               node_off[b] .. node_off[b+1]-1                              */
  const int32_t* kv_len;    /* [B] int32: prefix length L_b                                */
  const void* hidden;       /* [M][Hd] dtype: hidden state of every tree node              */
  const void* k_cache;      /* [B][Hkv][L_cap][D] dtype: rows 0..L_b-1 are the prefix, rows
                               L_b+j hold tree node j's own key                            */
  const void* v_cache;      /* [B][Hkv][L_cap][D] dtype, same layout for values            */
  const void* lm_head;      /* [V][Hd] dtype, row-major (nn.Linear weight layout)          */
  const int32_t* parent;    /* [M] int32, sequence-local: parent[root] = -1, else
                               0 <= parent[j] < j                                           */
  const int32_t* token;     /* [M] int32 draft token of each node in [0, V); the root's
                               entry is not checked                                        */
  const uint8_t* src;       /* [M] uint8 respec_src of each node                            */
  const float* draft_prob;  /* stochastic only: [M][V] float32, row i = the drafter's
                               distribution at node i (that its MODEL children were drawn
                               from), 16-byte aligned; NULL = every draft deterministic     */
  const float* uniform;     /* stochastic only (required): [M][2] float32 uniforms in [0,1):
                               [j][0] tests node j as a child, [j][1] draws at node j       */

  /* outputs (device) */
  float* attn_out;          /* [M][Hd] float32 attention output O, or NULL                 */
  void* x_out;              /* [M][Hd] dtype residual x = round(h + O) that feeds the LM
                               head (round to nearest even for bf16), or NULL              */
  float* logits;            /* [M][V] float32 logits z (required unless STOP_ATTN)         */
  float* max_logit;         /* [M] max_v z                                                  */
  float* lse;               /* [M] log sum_v exp z                                          */
  float* entropy;           /* [M] -sum_v p log p, nats (Eq. 1 inner sum)                  */
  int32_t* argmax;          /* [M] argmax_v z, smallest id on ties                          */
  int32_t* topk_id;         /* [M][topk_out] ids by (z desc, id asc)                        */
  float* topk_logprob;      /* [M][topk_out] log p of those ids                             */
  float* tok_logprob;       /* [M] log p_parent(t_j); 0 for roots                           */
  int32_t* tok_rank;        /* [M] rank of t_j in its parent's logits z_i, or NULL (not
                               computed; no decision depends on it, the TOPK flag holds
                               rank < k):  #{u : z_i[u] > z_i[t_j]} + #{u < t_j : z_i[u] ==
                               z_i[t_j]} on the float32 logits (0 = the argmax); -1 for
                               roots and for nodes without a valid parent or token        */
  uint8_t* flags;           /* [M] RESPEC_FLAG_* bits                                       */
  int32_t* leaf_acc_len;    /* [M] accepted length of each leaf's chain, -1 for inner nodes */
  int32_t* path;            /* [B][max_depth+1] sequence-local node ids of the accepted path,
                               root first, -1 padded                                        */
  int32_t* acc_len;         /* [B] accepted draft tokens (path length - 1), -1 on error    */
  int32_t* bonus;           /* [B] argmax at the last accepted node (the free token)       */
  int32_t* winner_leaf;     /* [B] sequence-local leaf whose chain won, -1 on error         */
  int32_t* seq_status;      /* [B] RESPEC_OK, RESPEC_ERR_TREE or RESPEC_ERR_TOKEN           */
  int32_t* sample;          /* stochastic, optional: [M] the residual draw at node i when no
                               child of i passes, else -1 (NULL = not written)             */

  void* stage_events;       /* optional host array of 4 hipEvent_t (profiling), NULL = none:
                               [0] start of the attention kernel, [1] end of the split
                               merge, [2] end of the LM head, [3] end of the vocab pass,
                               each taken from that kernel's own dispatch (a stage that
                               does not run records its event on the stream instead)      */
} respec_verify_args;

typedef struct respec_verify_plan respec_verify_plan;

/* Create a plan (host).  Validates the shape; *out receives the plan. */
respec_status respec_verify_create(const respec_verify_shape* shape, respec_verify_plan** out);

/* Destroy a plan (host).  NULL is ignored. */
void respec_verify_destroy(respec_verify_plan* plan);

/* Bytes of device workspace a step needs (host); 0 for a NULL plan. */
size_t respec_verify_workspace_bytes(const respec_verify_plan* plan);

/* Zero the workspace's completion counters (enqueued on stream).  Call once
 * after allocating a workspace; every completed step leaves them at zero. */
respec_status respec_verify_workspace_init(const respec_verify_plan* plan, void* workspace,
                                           void* stream);

/* Check one parent array on the host: parent[0] == -1, 0 <= parent[j] < j,
 * depth <= max_depth, 1 <= n <= RESPEC_MAX_NODES.  Returns RESPEC_OK,
 * RESPEC_ERR_TREE or RESPEC_ERR_NULL / RESPEC_ERR_SHAPE. */
respec_status respec_verify_check_tree(const int32_t* parent_host, int32_t n, int32_t max_depth);

/* Enqueue one verification step on stream (async).  workspace must hold
 * respec_verify_workspace_bytes(plan) bytes, 256-byte aligned, initialised by
 * respec_verify_workspace_init. */
respec_status respec_verify_step(const respec_verify_plan* plan, const respec_verify_args* args,
                                 void* workspace, void* stream);

/* Allocation-free form of respec_verify_step, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Same arguments, launches and results as
 * respec_verify_step, except that the workspace is not passed: the step uses a
 * static device array inside the library (RESPEC_NOALLOC_SCRATCH_BYTES, one per
 * GPU, held by every GPU the library runs on until the process ends).  The
 * first call on a device, with that device current, looks the array up and
 * clears its completion counters with a kernel enqueued on stream; no call
 * allocates or frees memory.  Returns RESPEC_ERR_SCRATCH, launching nothing,
 * when respec_verify_workspace_bytes(plan) exceeds
 * RESPEC_NOALLOC_SCRATCH_BYTES - 4 * RESPEC_NOALLOC_MAX_BATCH or the plan's
 * max_batch exceeds RESPEC_NOALLOC_MAX_BATCH; RESPEC_ERR_HIP when the array
 * cannot be looked up.  Every call on a GPU shares that GPU's array, which
 * keeps the last call's intermediates: calls that overlap on one GPU (other
 * streams or threads, without ordering between them) race, and the caller
 * must serialise them. */
respec_status respec_verify_step_noalloc(const respec_verify_plan* plan, const respec_verify_args* args,
                                         void* stream);

/* Static description of a status code. */
const char* respec_status_string(respec_status status);

#ifdef __cplusplus
}
#endif

#endif /* RESPEC_VERIFY_H */
