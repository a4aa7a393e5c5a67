/* respec_draft.h -- C ABI of the drafting side of one ReSpec decoding step (host).
 *
 * Retrieval-enhanced speculative decoding (ReSpec, arXiv 2511.01282) decides
 * per step whether to draft by retrieval from the context or with a model
 * drafter, and learns which retrieval positions are worth verifying.  This
 * header covers the host half of Algorithm 1 around the GPU verification step
 * of respec_verify.h:
 *
 *   Step 1  entropy-guided trigger (Section 3.2.1, Eq. 1-3)     respec_trigger_eval
 *   Step 2  retrieval positions from a suffix automaton         respec_sam_*
 *           EMA-scored filtering and top-n selection (Sec. 3.3,  respec_scores_*,
 *           Eq. 4-5)                                              respec_select
 *           BuildDraftTree: trie merge of the selected           respec_build_tree
 *           continuations into a parent-array draft tree
 *           EMA feedback after verification                      respec_scores_update
 *   Step 3  fallback to a model drafter (the caller's), strict verification
 *   append  accepted tokens to the context and the automaton    respec_draft_session_commit
 *
 * respec_draft_session_* composes the pieces in Algorithm 1's order for one
 * sequence; the pieces are exported too.
 *
 * Conventions
 *  - Every pointer is HOST memory owned by the caller; the library copies what
 *    it keeps.  Nothing here touches a GPU.
 *  - Token ids are int32 >= 0 (RESPEC_ERR_TOKEN otherwise).  Positions are
 *    0-based indices into the context: a retrieval position p is the index of
 *    the last token of an earlier occurrence of the key, and its continuation
 *    is context[p+1 ..].
 *  - Objects (automaton, score table, session) are not thread-safe; distinct
 *    objects may be used from distinct threads.
 *  - Functions return a status and leave outputs untouched on error, unless
 *    stated otherwise.  No exceptions cross this ABI; nothing is printed; an
 *    allocation failure returns RESPEC_ERR_CAPACITY.
 */
#ifndef RESPEC_DRAFT_H
#define RESPEC_DRAFT_H

#include <stddef.h>
#include <stdint.h>

#include "respec_verify.h"

#ifdef __cplusplus
extern "C" {
#endif

enum { RESPEC_DRAFT_MAX_SELECT = 16 };

/* ---------------------------------------------------------------- trigger */

/* Entropy-guided trigger (Section 3.2.1; Algorithm 1, Step 1). */
typedef struct {
  int32_t max_lookback;  /* l: longest retrieval key, >= 1 (the paper's experiments: 3) */
  float lambda_e;        /* length penalty of Eq. 2 (finite)                              */
  float theta_entropy;   /* trigger threshold, nats (the paper's experiments: 1.5)        */
} respec_trigger_params;

typedef struct {
  int32_t key_len;  /* k* of Eq. 3; 0 when no key length is available                  */
  float h_min;      /* H_{k*} of Eq. 1 (mean entropy of the key), NaN when key_len = 0   */
  float c_min;      /* C_{k*} of Eq. 2, NaN when key_len = 0                             */
  int32_t fire;     /* 1 iff key_len > 0 and h_min <= theta_entropy                     */
} respec_trigger_result;

/* Evaluate the trigger on the entropies of the context's most recent tokens.
 * entropy[0..n-1] (host, oldest first): entropy[i] is the Shannon entropy, in
 * nats, of the target distribution that produced context token i of the
 * window; entropy[n-1] belongs to the context's last token.  NaN marks a token
 * no distribution produced (the first prompt token).  For k = 1..l with the
 * last k entries all finite, H_k = (sum of the last k entries, added oldest
 * first in double) / k and C_k = H_k + lambda_e / k (double); k* is the
 * smallest k with the least C_k (Algorithm 1 replaces its best only on a
 * strictly smaller C).  n = 0 or a NaN last entry gives key_len = 0, fire = 0.
 * Errors: RESPEC_ERR_NULL (out, or entropy with n > 0), RESPEC_ERR_PARAM
 * (l < 1, non-finite lambda_e or theta_entropy), RESPEC_ERR_SHAPE (n < 0). */
respec_status respec_trigger_eval(const float* entropy, int32_t n, const respec_trigger_params* p,
                                  respec_trigger_result* out);

/* ------------------------------------------------------- suffix automaton */

/* Suffix automaton of the context (the index of Algorithm 1's retrieval and
 * of its SAM.Update).  It keeps its own copy of the context tokens. */
typedef struct respec_sam respec_sam;

respec_status respec_sam_create(respec_sam** out);
void respec_sam_destroy(respec_sam* sam);

/* Append tokens[0..n-1] to the context (n >= 0).  On RESPEC_ERR_TOKEN the
 * tokens before the first negative one have been appended. */
respec_status respec_sam_extend(respec_sam* sam, const int32_t* tokens, int32_t n);

/* Context length in tokens (0 for NULL). */
int64_t respec_sam_length(const respec_sam* sam);

/* Copy context tokens [start, start+n) to out.  RESPEC_ERR_SHAPE if the range
 * is not inside the context. */
respec_status respec_sam_text(const respec_sam* sam, int64_t start, int32_t n, int32_t* out);

/* Retrieval positions of key[0..k-1] (k >= 1): every position p with
 * context[p-k+1 .. p] == key and p < length-1 (an occurrence with at least one
 * following token; the context's own trailing occurrence has none), in
 * decreasing order.  The first min(cap, total) are written to pos_out (may be
 * NULL when cap = 0) and *n_total receives the total count.  An empty result
 * means the key is not contained (Algorithm 1's SAM.Contains is false).
 * The automaton keeps the positions of recent keys (up to 8 tokens) and brings
 * them up to date from the tokens appended since, so a query updates internal
 * state: concurrent queries on one automaton need external synchronisation. */
respec_status respec_sam_positions(const respec_sam* sam, const int32_t* key, int32_t k, int32_t* pos_out,
                                   int32_t cap, int32_t* n_total);

/* ------------------------------------------- EMA scores and selection */

/* Feedback-driven candidate selection (Section 3.3, Eq. 4-5; Algorithm 1). */
typedef struct {
  float alpha;        /* EMA update rate of Eq. 4, in [0, 1]                                 */
  float theta_score;  /* quality threshold: positions with S < theta_score are dropped       */
  float s0;           /* score of a position never scored before (the paper's example: 0.5)  */
  int32_t n_select;   /* candidates kept, 1..RESPEC_DRAFT_MAX_SELECT (the paper: 3)          */
} respec_select_params;

/* Score table S_pos, one double per scored position. */
typedef struct respec_scores respec_scores;

respec_status respec_scores_create(respec_scores** out);
void respec_scores_destroy(respec_scores* sc);

/* Score of position pos, or s0 if it has never been updated. */
double respec_scores_get(const respec_scores* sc, int32_t pos, double s0);

/* Number of positions with a stored score. */
int64_t respec_scores_size(const respec_scores* sc);

/* Threshold filtering and ranking: keep the positions with S_pos >=
 * theta_score (both in double), order them by S_pos descending, ties by
 * position descending (the more recent occurrence first), and write the first
 * min(n_select, kept) to sel_out[RESPEC_DRAFT_MAX_SELECT]; *n_sel receives the
 * count.  pos[0..n-1] must be distinct.  Errors: RESPEC_ERR_NULL,
 * RESPEC_ERR_SHAPE (n < 0 or a negative position), RESPEC_ERR_PARAM (parameters
 * out of range). */
respec_status respec_select(const respec_scores* sc, const int32_t* pos, int32_t n, const respec_select_params* p,
                            int32_t* sel_out, int32_t* n_sel);

/* EMA feedback (Eq. 4-5; Algorithm 1): for each i < n_sel,
 * R = (i == winner) ? (double)l_acc / l_draft[i] : 0, and
 * S <- (1 - alpha) * S + alpha * R in double (alpha widened from float), with
 * S starting at s0.  winner = -1 means no candidate won; otherwise
 * 0 <= winner < n_sel, l_draft[winner] >= 1 and 0 <= l_acc <= l_draft[winner]
 * (RESPEC_ERR_SHAPE otherwise; l_draft may be NULL when winner = -1).
 * sel[0..n_sel-1] must be distinct positions >= 0 (RESPEC_ERR_SHAPE). */
respec_status respec_scores_update(respec_scores* sc, const int32_t* sel, int32_t n_sel, int32_t winner,
                                   int32_t l_acc, const int32_t* l_draft, const respec_select_params* p);

/* -------------------------------------------------------- BuildDraftTree */

typedef struct {
  int32_t max_draft_len;  /* tokens taken from each continuation, >= 1                       */
  int32_t max_nodes;      /* tree nodes including the root, 2..RESPEC_MAX_NODES              */
} respec_tree_params;

/* BuildDraftTree (Algorithm 1): the root is the context's last token; the
 * continuation of candidate i is context[sel[i]+1 .. sel[i]+max_draft_len],
 * cut at the context's end; continuations are merged into a trie in the order
 * of sel (shared prefixes share nodes), nodes numbered in creation order so
 * that parent[j] < j; a new node is created only while the tree has fewer
 * than max_nodes nodes, which cuts later continuations short.  Outputs (host,
 * capacity max_nodes): parent[] (root -1), token[], src[] (root MODEL, every
 * other node RETRIEVED), *n_nodes; per candidate cand_end[i] (the node of its
 * last token in the tree, 0 if none fit) and cand_len[i] (its tokens in the
 * tree = depth of cand_end[i]).  Errors: RESPEC_ERR_NULL, RESPEC_ERR_PARAM,
 * RESPEC_ERR_SHAPE (empty context, n_sel outside 0..RESPEC_DRAFT_MAX_SELECT,
 * a position outside the context). */
respec_status respec_build_tree(const respec_sam* sam, const int32_t* sel, int32_t n_sel, const respec_tree_params* p,
                                int32_t* parent, int32_t* token, uint8_t* src, int32_t* n_nodes, int32_t* cand_end,
                                int32_t* cand_len);

/* ---------------------------------------------------------------- session */

/* Algorithm 1's host side for one sequence: context, automaton, entropy
 * history and score table. */
typedef struct {
  respec_trigger_params trigger;
  respec_select_params select;
  respec_tree_params tree;
} respec_draft_params;

typedef struct respec_draft_session respec_draft_session;

typedef struct {
  int32_t retrieved;          /* 1: the tree was built by retrieval (relaxed verification of its
                                 RETRIEVED nodes); 0: fall back to the model drafter (Step 3)  */
  respec_trigger_result trigger;
  int32_t n_positions;        /* |P|, retrieval positions of the key (0 if not triggered)       */
  int32_t n_selected;         /* |P_selected|                                                   */
  int32_t sel_pos[RESPEC_DRAFT_MAX_SELECT];
  int32_t cand_end[RESPEC_DRAFT_MAX_SELECT];
  int32_t cand_len[RESPEC_DRAFT_MAX_SELECT];
  int32_t n_nodes;            /* tree nodes written (1 = root only when not retrieved)          */
} respec_draft_result;

respec_status respec_draft_session_create(const respec_draft_params* p, respec_draft_session** out);
void respec_draft_session_destroy(respec_draft_session* s);

/* Append tokens to the context with the entropies of the target distributions
 * that produced them (entropy may be NULL: all NaN).  Used for the prompt. */
respec_status respec_draft_session_append(respec_draft_session* s, const int32_t* tokens, const float* entropy,
                                          int32_t n);

/* Steps 1-2 up to BuildDraftTree: evaluate the trigger on the context's last
 * l entropies; if it fires and the automaton holds the key, retrieve, filter,
 * select and build the tree into parent/token/src (capacity cap_nodes >=
 * tree.max_nodes).  Otherwise write the root alone and set retrieved = 0. The
 * session remembers the proposal for commit.  Errors: RESPEC_ERR_NULL,
 * RESPEC_ERR_SHAPE (empty context, cap_nodes too small). */
respec_status respec_draft_session_propose(respec_draft_session* s, int32_t* parent, int32_t* token, uint8_t* src,
                                           int32_t cap_nodes, respec_draft_result* out);

/* After verification of the proposed tree (or of the caller's model-drafted
 * tree after a proposal with retrieved = 0): token[] is the verified tree's
 * token array, path[0..acc_len] its accepted path (sequence-local node ids,
 * root first: respec_verify_step's path row), bonus the free token, and
 * entropy[] the per-node entropies of that step; token[] and entropy[] must
 * hold every node of the path.  If the proposal was
 * retrieved, the selected positions get their EMA update: the winner is the
 * first candidate, in selection order, whose chain holds path[acc_len], with
 * l_acc = acc_len and l_draft = its cand_len; the others get R = 0.  Then the
 * accepted tokens token[path[1..acc_len]] and the bonus are appended with the
 * entropies entropy[path[0..acc_len]] (Algorithm 1: X <- X + X_accepted and
 * SAM.Update).  Errors: RESPEC_ERR_NULL, RESPEC_ERR_SHAPE (acc_len < 0 or
 * a path entry < 0), RESPEC_ERR_TREE (for a retrieved proposal: a path that is
 * not a root-to-node chain of the proposed tree). */
respec_status respec_draft_session_commit(respec_draft_session* s, const int32_t* token, const int32_t* path,
                                          int32_t acc_len, int32_t bonus, const float* entropy);

/* Read-only views of a session's automaton and score table (owned by it). */
const respec_sam* respec_draft_session_sam(const respec_draft_session* s);
const respec_scores* respec_draft_session_scores(const respec_draft_session* s);

#ifdef __cplusplus
}
#endif

#endif /* RESPEC_DRAFT_H */
