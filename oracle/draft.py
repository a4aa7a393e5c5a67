"""Oracle of the drafting side of a ReSpec decoding step (TEST INFRASTRUCTURE ONLY).

Only ``tests/`` may import this module.  Plain Python loops, written from the
paper's definitions; it shares no code with the library (whose drafting side
is C++ with a suffix automaton) and uses no index structure at all: retrieval
positions are found by scanning the whole context.

Paper: "When, What, and How: Rethinking Retrieval-Enhanced Speculative
Decoding" (ReSpec, arXiv 2511.01282).

  trigger_eval   Section 3.2.1, Eq. 1-3 and Algorithm 1 (Step 1)
  positions      Algorithm 1: SAM.Contains / SAM.RetrievePositions, by definition
  select         Section 3.3 (threshold filtering, ranking and top-n selection)
  ema_update     Section 3.3, Eq. 4-5 and Algorithm 1's feedback loop
  build_tree     Algorithm 1: BuildDraftTree (trie merge of the continuations)
  Session        Algorithm 1 for one sequence, the verification left to the caller

Readings of the paper taken here (listed with the others in the repository's
design notes):
  - Eq. 1 averages the entropies of the distributions that produced the key's
    own tokens (the latest ones available when the trigger runs); a token with
    no producing distribution (NaN) ends the usable key lengths;
  - k* is the smallest k with the least C_k (Algorithm 1 replaces only on a
    strictly smaller C); the trigger fires when H_{k*} <= theta (inclusive);
  - a key is "contained" when it also occurs earlier with a following token;
    the positions are those occurrences' last-token indices;
  - equal scores rank the more recent position first;
  - only the selected positions are updated; the winner is the first selected
    candidate whose chain holds the last accepted node, with R = accepted
    length / its length in the tree, every other selected one gets R = 0;
  - continuations hold at most max_draft_len tokens, the tree at most
    max_nodes nodes, filled in selection order.

Parity pins (tests): the trigger against closed forms (constant entropies,
lambda = 0 against cumulative means), retrieval against a regular-expression
scan, the EMA against its closed form, the tree against the set of distinct
prefixes, and the whole loop under strict verification against plain greedy
decoding.
"""
from __future__ import annotations

import math

SRC_MODEL, SRC_RETRIEVED = 0, 1


def trigger_eval(entropy, max_lookback, lambda_e, theta_entropy):
    """Eq. 1-3 over the entropies of the context's last tokens (oldest first).

    Returns (key_len, h_min, c_min, fire); key_len = 0 when no key is usable.
    """
    n = len(entropy)
    c_min, h_best, key_len = math.inf, math.inf, 0
    for k in range(1, max_lookback + 1):           # Algorithm 1, Step 1
        if k > n:
            break
        window = [float(entropy[i]) for i in range(n - k, n)]
        if any(not math.isfinite(v) for v in window):
            break
        h_k = 0.0
        for v in window:                            # Eq. 1: mean entropy of the key's tokens
            h_k += v
        h_k = h_k / k
        c_k = h_k + float(lambda_e) / k             # Eq. 2
        if key_len == 0 or c_k < c_min:             # Eq. 3: arg min, first minimum kept
            c_min, h_best, key_len = c_k, h_k, k
    if key_len == 0:
        return 0, math.nan, math.nan, False
    return key_len, h_best, c_min, h_best <= float(theta_entropy)


def positions(text, key):
    """Every p < len(text)-1 with text[p-k+1..p] == key, most recent first."""
    k, n = len(key), len(text)
    out = []
    for p in range(k - 1, n - 1):
        if all(text[p - k + 1 + i] == key[i] for i in range(k)):
            out.append(p)
    out.reverse()
    return out


def select(scores, pos, alpha, theta_score, s0, n_select):
    """Threshold filtering, then the n_select best by score (ties: more recent first)."""
    kept = [(scores.get(p, float(s0)), p) for p in pos]
    kept = [(s, p) for (s, p) in kept if s >= float(theta_score)]
    kept.sort(key=lambda sp: (-sp[0], -sp[1]))
    return [p for (_, p) in kept[:n_select]]


def ema_update(scores, sel, winner, l_acc, l_draft, alpha, s0):
    """Eq. 4-5 for every selected position (dict scores updated in place)."""
    a = float(alpha)
    for i, p in enumerate(sel):
        r = float(l_acc) / float(l_draft[i]) if i == winner else 0.0      # Eq. 5
        s = scores.get(p, float(s0))
        scores[p] = (1.0 - a) * s + a * r                                   # Eq. 4


def build_tree(text, sel, max_draft_len, max_nodes):
    """BuildDraftTree: the root is the last token; continuations merged as a trie.

    Returns (parent, token, src, cand_end, cand_len) as lists.
    """
    parent, token, src = [-1], [text[-1]], [SRC_MODEL]
    children = {0: []}
    cand_end, cand_len = [], []
    for p in sel:
        cont = text[p + 1: min(len(text), p + 1 + max_draft_len)]
        node, depth = 0, 0
        for t in cont:
            nxt = None
            for c in children[node]:
                if token[c] == t:
                    nxt = c
                    break
            if nxt is None:
                if len(parent) >= max_nodes:
                    break
                nxt = len(parent)
                parent.append(node)
                token.append(t)
                src.append(SRC_RETRIEVED)
                children[node].append(nxt)
                children[nxt] = []
            node, depth = nxt, depth + 1
        cand_end.append(node)
        cand_len.append(depth)
    return parent, token, src, cand_end, cand_len


class Session:
    """Algorithm 1's host side for one sequence, in the paper's order."""

    def __init__(self, max_lookback=3, lambda_e=0.5, theta_entropy=1.5, alpha=0.5, theta_score=0.1, s0=0.5,
                 n_select=3, max_draft_len=20, max_nodes=61):
        self.l, self.lam, self.theta = max_lookback, lambda_e, theta_entropy
        self.alpha, self.theta_score, self.s0, self.n_select = alpha, theta_score, s0, n_select
        self.max_draft_len, self.max_nodes = max_draft_len, max_nodes
        self.text, self.entropy, self.scores = [], [], {}
        self.last = None

    def append(self, tokens, entropy=None):
        for i, t in enumerate(tokens):
            self.text.append(int(t))
            self.entropy.append(math.nan if entropy is None else float(entropy[i]))

    def propose(self):
        """Returns a dict: retrieved, trigger, n_positions, selected, tree (parent, token, src), cand_end, cand_len."""
        n = len(self.text)
        w = min(n, self.l)
        trig = trigger_eval(self.entropy[n - w:], self.l, self.lam, self.theta)
        key_len, _, _, fire = trig
        pos = positions(self.text, self.text[n - key_len:]) if fire else []
        res = dict(retrieved=False, trigger=trig, n_positions=len(pos), selected=[], cand_end=[], cand_len=[],
                   parent=[-1], token=[self.text[-1]], src=[SRC_MODEL])
        if fire and pos:
            sel = select(self.scores, pos, self.alpha, self.theta_score, self.s0, self.n_select)
            if sel:
                parent, token, src, ce, cl = build_tree(self.text, sel, self.max_draft_len, self.max_nodes)
                res.update(retrieved=True, selected=sel, parent=parent, token=token, src=src, cand_end=ce,
                           cand_len=cl)
        self.last = res
        return res

    def commit(self, token, path, acc_len, bonus, entropy):
        r = self.last
        if r is not None and r["retrieved"]:
            tip = path[acc_len]
            winner = -1
            for c, end in enumerate(r["cand_end"]):
                v = end
                chain = []
                while v >= 0:
                    chain.append(v)
                    v = r["parent"][v]
                if tip in chain:
                    winner = c
                    break
            if winner >= 0 and r["cand_len"][winner] < 1:
                winner = -1
            ema_update(self.scores, r["selected"], winner, acc_len, r["cand_len"], self.alpha, self.s0)
        for j in range(1, acc_len + 1):
            self.text.append(int(token[path[j]]))
            self.entropy.append(float(entropy[path[j - 1]]))
        self.text.append(int(bonus))
        self.entropy.append(float(entropy[path[acc_len]]))
        self.last = None
