/* respec_oracle.c -- plain, slow CPU oracle for one draft-tree verification step.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no code with
 * the GPU path.
 *
 * Paper: "When, What, and How: Rethinking Retrieval-Enhanced Speculative
 * Decoding" (ReSpec, arXiv 2511.01282).  Each function cites the passage it
 * follows.  Everything is accumulated in double.  Inputs arrive as the exact
 * float32 or bf16 bit patterns the GPU receives (dtype 0 = float32, 1 = bf16
 * stored as uint16) and are widened to double without loss.
 *
 * Readings of the paper that this oracle takes where the text is silent or
 * ambiguous (each is listed in the design notes of the repository):
 *  - entropy is in nats, temperature 1 (Eq. 1);
 *  - strict verification is greedy: the draft token must equal the target's
 *    argmax at its parent (Section 4.1, implementation details);
 *  - a node passes the relaxed check if it is a greedy match or, for a
 *    retrieved node, if its token is in TopK_k of the parent distribution and
 *    its log-probability gap to the top-1 token is <= tau (Eq. 6-7);
 *  - the look-ahead tolerance procedure (Section 3.4) is applied to every
 *    root-to-leaf chain of the tree; the longest result wins, ties going to
 *    the path whose last accepted node has the smallest index;
 *  - ties in argmax and top-k go to the smallest token id;
 *  - decisions that turn logits into integers (argmax, rank, the tau test)
 *    are taken on logits rounded to float32, the precision the GPU kernel
 *    stores them in.
 *
 *  - stochastic verification (drafter outputs verified by lossless
 *    speculative sampling, Section 3.4) tries a node's children in index
 *    order, each against the residual left by the rejected ones; a retrieved
 *    child is a deterministic draft (one-hot draft distribution).
 *
 * Parity pins (tests): chain trees against textbook causal attention, star
 * trees against decode attention, logits against a library GEMM, entropy and
 * log-sum-exp against library routines and closed forms, top-k against a full
 * stable sort, hand-worked look-ahead cases, brute-force path enumeration.
 * The look-ahead reading itself has no worked example in the paper: parity of
 * that step is unpinned beyond the hand-worked cases derived from the prose.
 * Stochastic verification: hand-worked acceptance probabilities and residual
 * draws, Monte Carlo losslessness (the emitted token follows the target
 * distribution), a drafter equal to the target, and the vanishing-temperature
 * limit against greedy verification.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_F32 0
#define ORACLE_BF16 1
#define SRC_RETRIEVED 1

/* flag bits, per node (about the node's own draft token) */
#define FLAG_GREEDY 1u   /* token == argmax of the parent's distribution       */
#define FLAG_TOPK 2u     /* token in TopK_k of the parent's distribution       */
#define FLAG_TAU 4u      /* log p(top1) - log p(token) <= tau                   */
#define FLAG_RELAXED 8u  /* retrieved and TOPK and TAU (Eq. 6-7)                */
#define FLAG_ON_PATH 16u /* node is on the accepted path (root included)        */

/* Number of OpenMP threads the oracle's parallel loops use. */
int32_t respec_oracle_threads(void) { return (int32_t)omp_get_max_threads(); }

/* Set that number (for timing the oracle on one thread and on all of them). */
void respec_oracle_set_threads(int32_t n) { omp_set_num_threads(n > 0 ? n : 1); }

static double bf16_to_double(uint16_t b) {
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, 4);
    return (double)f;
}

static double load(int32_t dtype, const void* base, int64_t i) {
    if (dtype == ORACLE_BF16) return bf16_to_double(((const uint16_t*)base)[i]);
    return (double)((const float*)base)[i];
}

/* ------------------------------------------------------------------------ */
/* Tree (Algorithm 1, BuildDraftTree / RelaxedVerify; Section 3.5).
 * parent[0] = -1 marks the root; every other node's parent precedes it.
 * Outputs depth (root = 0), the ancestor-or-self matrix anc[i*n + j] = 1 iff
 * j is on the root-to-i chain, and leaf flags.  Returns 0, or
 * 1 bad root, 2 bad parent index, 3 depth above max_depth, 4 n < 1.        */
int respec_oracle_tree(const int32_t* parent, int32_t n, int32_t max_depth,
                       int32_t* depth, uint8_t* anc, uint8_t* is_leaf) {
    if (n < 1) return 4;
    if (parent[0] != -1) return 1;
    for (int32_t j = 1; j < n; ++j)
        if (parent[j] < 0 || parent[j] >= j) return 2;
    memset(anc, 0, (size_t)n * (size_t)n);
    for (int32_t i = 0; i < n; ++i) {
        is_leaf[i] = 1;
        depth[i] = 0;
    }
    for (int32_t i = 0; i < n; ++i) {
        int32_t a = i;
        while (a >= 0) {
            anc[(size_t)i * n + a] = 1;
            if (a != i) depth[i] += 1;
            a = (a == 0) ? -1 : parent[a];
        }
        if (i > 0) is_leaf[parent[i]] = 0;
        if (depth[i] > max_depth) return 3;
    }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Tree-masked attention of the draft nodes against the KV cache (the
 * target's parallel verification forward, Section 3.5 / Algorithm 1;
 * reduced here to one attention layer).  The query of node i, head h is the
 * node's hidden state viewed as heads: q = hidden[i][h*D .. h*D+D).  KV head
 * g = h / (Hq/Hkv).  Node i sees every prefix row p < L and the tree row
 * L + a for every ancestor-or-self a of i.  Scores are <q, k_p> / sqrt(D);
 * the output is the softmax-weighted mean of the visible V rows.
 * k_seq/v_seq point at this sequence's [Hkv][kv_cap][D] block.
 * rows lists the node indices to compute; out is [n_rows][Hq*D].           */
void respec_oracle_attention(int32_t dtype, const void* hidden, int32_t hidden_size,
                             const void* k_seq, const void* v_seq, int32_t kv_cap,
                             int32_t kv_len, int32_t n_nodes, const uint8_t* anc,
                             int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                             const int32_t* rows, int32_t n_rows, double* out) {
    const int32_t group = n_q_heads / n_kv_heads;
    const double scale = 1.0 / sqrt((double)head_dim);
    const int64_t total = (int64_t)n_rows * n_q_heads;
#pragma omp parallel
    {
        int32_t n_vis_max = kv_len + n_nodes;
        double* score = (double*)malloc(sizeof(double) * (size_t)n_vis_max);
        int32_t* pos = (int32_t*)malloc(sizeof(int32_t) * (size_t)n_vis_max);
        double* q = (double*)malloc(sizeof(double) * (size_t)head_dim);
#pragma omp for schedule(dynamic)
        for (int64_t t = 0; t < total; ++t) {
            int32_t r = (int32_t)(t / n_q_heads), h = (int32_t)(t % n_q_heads);
            int32_t i = rows[r], g = h / group;
            for (int32_t d = 0; d < head_dim; ++d)
                q[d] = load(dtype, hidden, (int64_t)i * hidden_size + (int64_t)h * head_dim + d);
            int32_t nv = 0;
            for (int32_t p = 0; p < kv_len; ++p) pos[nv++] = p;
            for (int32_t a = 0; a < n_nodes; ++a)
                if (anc[(size_t)i * n_nodes + a]) pos[nv++] = kv_len + a;
            double mx = -INFINITY;
            for (int32_t s = 0; s < nv; ++s) {
                int64_t base = ((int64_t)g * kv_cap + pos[s]) * head_dim;
                double dot = 0.0;
                for (int32_t d = 0; d < head_dim; ++d) dot += q[d] * load(dtype, k_seq, base + d);
                score[s] = dot * scale;
                if (score[s] > mx) mx = score[s];
            }
            double denom = 0.0;
            for (int32_t s = 0; s < nv; ++s) {
                score[s] = exp(score[s] - mx);
                denom += score[s];
            }
            double* o = out + (int64_t)r * n_q_heads * head_dim + (int64_t)h * head_dim;
            for (int32_t d = 0; d < head_dim; ++d) o[d] = 0.0;
            for (int32_t s = 0; s < nv; ++s) {
                int64_t base = ((int64_t)g * kv_cap + pos[s]) * head_dim;
                double w = score[s] / denom;
                for (int32_t d = 0; d < head_dim; ++d) o[d] += w * load(dtype, v_seq, base + d);
            }
        }
        free(score);
        free(pos);
        free(q);
    }
}

/* ------------------------------------------------------------------------ */
/* Round d to the nearest number with `sig` significant bits, ties to even:
 * d = m 2^e with 1/2 <= |m| < 1, so the spacing of such numbers at d is
 * 2^(e - sig); below the normal range the spacing stays 2^min_exp.  d / q and
 * rint(.) q are exact, and rint rounds half to even.  float32 is (24, -149),
 * bf16 (8, -133); the values here stay far inside both ranges.             */
static double round_sig(double d, int sig, int min_exp) {
    if (d == 0.0 || !isfinite(d)) return d;
    int e;
    frexp(d, &e);
    int qe = e - sig;
    if (qe < min_exp) qe = min_exp;
    double q = ldexp(1.0, qe);
    return rint(d / q) * q;
}

/* Residual and rounding point of the one-layer proxy: x = round(h + O), the
 * exact sum h + O (in double) rounded once to the workload dtype, round to
 * nearest even.  x is returned widened to double (exactly representable).  */
void respec_oracle_residual(int32_t dtype, const void* hidden, const double* attn,
                            int64_t count, double* x) {
    for (int64_t i = 0; i < count; ++i) {
        double s = load(dtype, hidden, i) + attn[i];
        x[i] = dtype == ORACLE_BF16 ? round_sig(s, 8, -133) : round_sig(s, 24, -149);
    }
}

/* ------------------------------------------------------------------------ */
/* LM head: z[r][v] = sum_c x[r][c] * W[v][c]  (W is [V][Hd], row-major).
 * The target distribution P_t is softmax(z) (Section 3.2.1).               */
void respec_oracle_logits(int32_t dtype, const double* x, int32_t n_rows, int32_t hidden_size,
                          const void* w, int32_t vocab, double* z) {
    const int64_t total = (int64_t)n_rows * vocab;
#pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < total; ++t) {
        int32_t r = (int32_t)(t / vocab), v = (int32_t)(t % vocab);
        double acc = 0.0;
        for (int32_t c = 0; c < hidden_size; ++c)
            acc += x[(int64_t)r * hidden_size + c] * load(dtype, w, (int64_t)v * hidden_size + c);
        z[t] = acc;
    }
}

/* ------------------------------------------------------------------------ */
/* Per-row statistics of the target distribution p = softmax(z):
 *   max logit, argmax (smallest id on ties), log-sum-exp,
 *   Shannon entropy -sum_v p(v) log p(v) in nats (Eq. 1, inner sum),
 *   the topk_out most likely tokens ordered by (logit desc, id asc) with
 *   their log-probabilities.  z is the float32 logit row.                   */
static const float* g_sort_row;
static int cmp_desc(const void* a, const void* b) {
    int32_t ia = *(const int32_t*)a, ib = *(const int32_t*)b;
    float za = g_sort_row[ia], zb = g_sort_row[ib];
    if (za > zb) return -1;
    if (za < zb) return 1;
    return (ia > ib) - (ia < ib);
}

void respec_oracle_row_stats(const float* z, int32_t n_rows, int32_t vocab, int32_t topk_out,
                             double* max_logit, int32_t* argmax, double* lse, double* entropy,
                             int32_t* topk_id, double* topk_logprob) {
    int32_t* idx = (int32_t*)malloc(sizeof(int32_t) * (size_t)vocab);
    for (int32_t r = 0; r < n_rows; ++r) {
        const float* row = z + (int64_t)r * vocab;
        double mx = -INFINITY;
        int32_t am = 0;
        for (int32_t v = 0; v < vocab; ++v)
            if ((double)row[v] > mx) { mx = row[v]; am = v; }
        double s = 0.0;
        for (int32_t v = 0; v < vocab; ++v) s += exp((double)row[v] - mx);
        double l = mx + log(s);
        double h = 0.0;
        for (int32_t v = 0; v < vocab; ++v) {
            double lp = (double)row[v] - l;
            double p = exp(lp);
            h -= p * lp;
        }
        max_logit[r] = mx;
        argmax[r] = am;
        lse[r] = l;
        entropy[r] = h;
        for (int32_t v = 0; v < vocab; ++v) idx[v] = v;
        g_sort_row = row;
        qsort(idx, (size_t)vocab, sizeof(int32_t), cmp_desc);
        for (int32_t k = 0; k < topk_out; ++k) {
            topk_id[(int64_t)r * topk_out + k] = k < vocab ? idx[k] : -1;
            topk_logprob[(int64_t)r * topk_out + k] = k < vocab ? (double)row[idx[k]] - l : -INFINITY;
        }
    }
    free(idx);
}

/* rank of token t in row z: #{u : z_u > z_t} + #{u < t : z_u == z_t}        */
int32_t respec_oracle_rank(const float* row, int32_t vocab, int32_t t) {
    int32_t r = 0;
    for (int32_t u = 0; u < vocab; ++u)
        if (row[u] > row[t] || (row[u] == row[t] && u < t)) ++r;
    return r;
}

/* ------------------------------------------------------------------------ */
/* Per-node acceptance predicates for one sequence (Section 3.4).
 * For a non-root node j with parent i and draft token t = token[j]:
 *   GREEDY  t == argmax_i  (strict, greedy verification)
 *   TOPK    t in TopK_k(p_i), i.e. rank_i(t) < k        (Eq. 6)
 *   TAU     log p_i(top1) - log p_i(t) <= tau           (Eq. 7; the log-sum-exp
 *           cancels, so the test is z_i[argmax] - z_i[t] <= tau)
 *   RELAXED src_j == retrieved and TOPK and TAU
 * tok_logprob[j] = log p_i(t); tok_rank[j] = rank_i(t).  The root has no
 * predicate (0 flags, logprob 0, rank -1).  z is [n][V] float32.            */
void respec_oracle_node_flags(int32_t n, const int32_t* parent, const int32_t* token,
                              const uint8_t* src, const float* z, int32_t vocab,
                              const int32_t* argmax, const double* lse, int32_t topk, float tau,
                              uint8_t* flags, double* tok_logprob, int32_t* tok_rank) {
    flags[0] = 0;
    tok_logprob[0] = 0.0;
    tok_rank[0] = -1;
    for (int32_t j = 1; j < n; ++j) {
        int32_t i = parent[j], t = token[j];
        const float* row = z + (int64_t)i * vocab;
        uint8_t f = 0;
        int32_t rank = respec_oracle_rank(row, vocab, t);
        if (t == argmax[i]) f |= FLAG_GREEDY;
        if (rank < topk) f |= FLAG_TOPK;
        if ((double)row[argmax[i]] - (double)row[t] <= (double)tau) f |= FLAG_TAU;
        if (src[j] == SRC_RETRIEVED && (f & FLAG_TOPK) && (f & FLAG_TAU)) f |= FLAG_RELAXED;
        flags[j] = f;
        tok_logprob[j] = (double)row[t] - lse[i];
        tok_rank[j] = rank;
    }
}

/* ------------------------------------------------------------------------ */
/* Look-ahead tolerance along one candidate chain u_1..u_d (Section 3.4).
 * greedy[s] / ok[s] describe u_{s+1}: ok = greedy or relaxed pass.
 *   l0   = longest greedy prefix;  current = last = l0
 *   up to phi attempts, while current < d:
 *     relaxed check on u_{current+1}; on failure stop;
 *     xi = run of greedy matches starting at u_{current+2};
 *     if xi >= m: last = current + 1 + xi, current = last
 *     else        current = current + 1
 *   accepted length = last.                                                 */
int32_t respec_oracle_lookahead(int32_t d, const uint8_t* greedy, const uint8_t* ok,
                                int32_t m, int32_t phi) {
    int32_t l0 = 0;
    while (l0 < d && greedy[l0]) ++l0;
    int32_t current = l0, last = l0;
    for (int32_t attempt = 0; attempt < phi && current < d; ++attempt) {
        if (!ok[current]) break;
        int32_t xi = 0;
        while (current + 1 + xi < d && greedy[current + 1 + xi]) ++xi;
        if (xi >= m) {
            last = current + 1 + xi;
            current = last;
        } else {
            current = current + 1;
        }
    }
    return last;
}

/* ------------------------------------------------------------------------ */
/* Winner over a tree (Algorithm 1, RelaxedVerify -> X_accepted, p_winner).
 * Every leaf's root-to-leaf chain gets its look-ahead accepted length.  The
 * accepted path is the longest; ties go to the chain whose last accepted node
 * has the smallest index.  Outputs: leaf_acc_len[n] (-1 for inner nodes),
 * path[max_depth+1] (node ids, -1 padded), *acc_len, *bonus (argmax at the
 * last accepted node), *winner_leaf, and FLAG_ON_PATH in flags.
 * Requires a tree validated by respec_oracle_tree.                          */
void respec_oracle_path(int32_t n, const int32_t* parent, const uint8_t* is_leaf,
                        const int32_t* depth, uint8_t* flags, const int32_t* argmax,
                        int32_t max_depth, int32_t m, int32_t phi, int32_t* leaf_acc_len,
                        int32_t* path, int32_t* acc_len, int32_t* bonus, int32_t* winner_leaf) {
    int32_t* chain = (int32_t*)malloc(sizeof(int32_t) * (size_t)(max_depth + 1));
    uint8_t* g = (uint8_t*)malloc((size_t)max_depth + 1);
    uint8_t* ok = (uint8_t*)malloc((size_t)max_depth + 1);
    int32_t best = -1, best_end = n, best_leaf = -1;
    for (int32_t leaf = 0; leaf < n; ++leaf) {
        leaf_acc_len[leaf] = -1;
        if (!is_leaf[leaf]) continue;
        int32_t d = depth[leaf];
        int32_t a = leaf;
        for (int32_t s = d; s >= 1; --s) {  /* chain[s-1] = u_s */
            chain[s - 1] = a;
            a = parent[a];
        }
        for (int32_t s = 0; s < d; ++s) {
            g[s] = (flags[chain[s]] & FLAG_GREEDY) != 0;
            ok[s] = g[s] || (flags[chain[s]] & FLAG_RELAXED) != 0;
        }
        int32_t acc = respec_oracle_lookahead(d, g, ok, m, phi);
        leaf_acc_len[leaf] = acc;
        int32_t end = acc == 0 ? 0 : chain[acc - 1];
        if (acc > best || (acc == best && end < best_end)) {
            best = acc;
            best_end = end;
            best_leaf = leaf;
        }
    }
    for (int32_t s = 0; s <= max_depth; ++s) path[s] = -1;
    int32_t a = best_end;
    for (int32_t s = best; s >= 0; --s) {
        path[s] = a;
        flags[a] |= FLAG_ON_PATH;
        a = (a == 0) ? -1 : parent[a];
    }
    *acc_len = best;
    *bonus = argmax[best_end];
    *winner_leaf = best_leaf;
    free(chain);
    free(g);
    free(ok);
}

/* ------------------------------------------------------------------------ */
/* Stochastic (lossless) verification.  Section 3.4 verifies drafter outputs
 * with standard lossless speculative sampling: a draft token t drawn from the
 * drafter's distribution q is accepted with probability min(1, p(t) / q(t))
 * under the target's distribution p; on rejection the next token is drawn
 * from the residual norm(max(p - q, 0)).  A tree node with several children
 * tries them in order (recursive rejection over siblings, the multi-draft
 * form of the same rule): child k is tested against the residual r left by
 * the rejection of children 1..k-1, and each rejection replaces r by
 * norm(max(r - q_k, 0)).  A model-drafted child uses the drafter's
 * distribution at its parent; a retrieved child is a deterministic draft,
 * q_k = one-hot at its token.  Random numbers are inputs: u_acc[k] decides
 * child k (accept iff u < a), u_res the residual draw (inverse CDF: the
 * smallest v whose cumulative residual mass exceeds u_res times the total).
 * Everything in double; p = softmax(z / T) from the float32 logits.
 *
 * One node: returns the index of the first accepted child, or -1 when every
 * child is rejected, in which case *sample receives the residual draw (else
 * -1).  q_row may be NULL: every child is then a deterministic draft.
 * If a rejection leaves no residual mass (r = q_k), r is kept as it was.   */
int32_t respec_oracle_stoch_node(int32_t vocab, const float* z_row, float temperature, const float* q_row,
                                 int32_t n_child, const int32_t* child_tok, const uint8_t* child_model,
                                 const float* u_acc, float u_res, int32_t* sample) {
    double* r = (double*)malloc(sizeof(double) * (size_t)vocab);
    const double T = (double)temperature;
    double m = -INFINITY, s = 0.0;
    for (int32_t v = 0; v < vocab; ++v)
        if ((double)z_row[v] > m) m = (double)z_row[v];
    for (int32_t v = 0; v < vocab; ++v) {
        r[v] = exp(((double)z_row[v] - m) / T);
        s += r[v];
    }
    for (int32_t v = 0; v < vocab; ++v) r[v] /= s;          /* p = softmax(z / T) */
    int32_t accepted = -1;
    for (int32_t k = 0; k < n_child && accepted < 0; ++k) {
        const int32_t t = child_tok[k];
        const int model = child_model[k] && q_row != NULL;
        const double qt = model ? (double)q_row[t] : 1.0;
        const double rt = r[t];
        const double a = qt > 0.0 ? (rt / qt < 1.0 ? rt / qt : 1.0) : (rt > 0.0 ? 1.0 : 0.0);
        if ((double)u_acc[k] < a) {
            accepted = k;
            break;
        }
        double z = 0.0;
        for (int32_t v = 0; v < vocab; ++v) {
            const double qv = model ? (double)q_row[v] : (v == t ? 1.0 : 0.0);
            const double d = r[v] - qv;
            z += d > 0.0 ? d : 0.0;
        }
        if (z > 0.0)
            for (int32_t v = 0; v < vocab; ++v) {
                const double qv = model ? (double)q_row[v] : (v == t ? 1.0 : 0.0);
                const double d = r[v] - qv;
                r[v] = d > 0.0 ? d / z : 0.0;
            }
    }
    *sample = -1;
    if (accepted < 0) {
        double total = 0.0;
        for (int32_t v = 0; v < vocab; ++v) total += r[v];
        const double thr = (double)u_res * total;
        double c = 0.0;
        int32_t last_pos = 0;
        for (int32_t v = 0; v < vocab; ++v) {
            if (r[v] > 0.0) last_pos = v;
            c += r[v];
            if (c > thr) {
                *sample = v;
                break;
            }
        }
        if (*sample < 0) *sample = last_pos;
    }
    free(r);
    return accepted;
}

/* Stochastic verification of one sequence's tree.  Children of a node are
 * tried in node-index order.  Per node i: first_acc[i] = the first accepted
 * child (global to the sequence, -1 if none), sample[i] = the residual draw
 * when no child is accepted (else -1), acc_bit[j] = 1 iff j is the first
 * accepted child of its parent.  The walk starts at the root and moves to the
 * first accepted child until none is: path = the walked nodes (root first,
 * -1 padded to max_depth+1), acc_len = their count - 1, bonus = the residual
 * draw at the last one, winner_leaf = the smallest leaf whose chain holds the
 * last one, leaf_acc[l] = the number of walked non-root nodes on leaf l's
 * chain (-1 for inner nodes).  u holds two uniforms per node: [j][0] tests
 * node j as a child, [j][1] draws at node j.  q is [n][V] (row i: the
 * drafter's distribution at node i) or NULL.  Returns 0, or 1 for a tree
 * that respec_oracle_tree rejects (outputs untouched).                       */
int respec_oracle_stochastic(int32_t n, const int32_t* parent, const int32_t* token, const uint8_t* src,
                             const float* z32, int32_t vocab, const float* q, const float* u, float temperature,
                             int32_t max_depth, int32_t* first_acc, int32_t* sample, uint8_t* acc_bit,
                             int32_t* path, int32_t* acc_len, int32_t* bonus, int32_t* winner_leaf,
                             int32_t* leaf_acc) {
    int32_t* depth = (int32_t*)malloc(sizeof(int32_t) * (size_t)n);
    uint8_t* anc = (uint8_t*)malloc((size_t)n * (size_t)n);
    uint8_t* is_leaf = (uint8_t*)malloc((size_t)n);
    if (respec_oracle_tree(parent, n, max_depth, depth, anc, is_leaf) != 0) {
        free(depth);
        free(anc);
        free(is_leaf);
        return 1;
    }
    int32_t* kids = (int32_t*)malloc(sizeof(int32_t) * (size_t)n);
    int32_t* ktok = (int32_t*)malloc(sizeof(int32_t) * (size_t)n);
    uint8_t* kmodel = (uint8_t*)malloc((size_t)n);
    float* kuacc = (float*)malloc(sizeof(float) * (size_t)n);
    for (int32_t j = 0; j < n; ++j) acc_bit[j] = 0;
    for (int32_t i = 0; i < n; ++i) {
        int32_t nk = 0;
        for (int32_t j = i + 1; j < n; ++j)
            if (parent[j] == i) {
                kids[nk] = j;
                ktok[nk] = token[j];
                kmodel[nk] = src[j] != SRC_RETRIEVED;
                kuacc[nk] = u[2 * (size_t)j];
                ++nk;
            }
        const int32_t k = respec_oracle_stoch_node(vocab, z32 + (size_t)i * vocab, temperature,
                                                   q ? q + (size_t)i * vocab : NULL, nk, ktok, kmodel, kuacc,
                                                   u[2 * (size_t)i + 1], &sample[i]);
        first_acc[i] = k >= 0 ? kids[k] : -1;
        if (k >= 0) acc_bit[kids[k]] = 1;
    }
    /* the walk */
    uint8_t* walked = (uint8_t*)calloc((size_t)n, 1);
    for (int32_t d = 0; d <= max_depth; ++d) path[d] = -1;
    int32_t cur = 0, len = 0;
    walked[0] = 1;
    path[0] = 0;
    while (first_acc[cur] >= 0) {
        cur = first_acc[cur];
        walked[cur] = 1;
        path[++len] = cur;
    }
    *acc_len = len;
    *bonus = sample[cur];
    *winner_leaf = -1;
    for (int32_t l = 0; l < n; ++l) {
        if (!is_leaf[l]) {
            leaf_acc[l] = -1;
            continue;
        }
        int32_t c = 0;
        for (int32_t a = 1; a < n; ++a)
            if (anc[(size_t)l * n + a] && walked[a]) ++c;
        leaf_acc[l] = c;
        if (*winner_leaf < 0 && anc[(size_t)l * n + cur]) *winner_leaf = l;
    }
    free(walked);
    free(kids);
    free(ktok);
    free(kmodel);
    free(kuacc);
    free(depth);
    free(anc);
    free(is_leaf);
    return 0;
}
