"""Pins of the drafting-side oracle (oracle/draft.py) against what the paper and
the mathematics fix: hand-worked trigger cases (Eq. 1-3), closed forms, a
regular-expression scan for retrieval, the EMA's closed form (Eq. 4-5), the set
of distinct prefixes for BuildDraftTree, and, for the whole loop of
Algorithm 1, the losslessness of strict verification: speculative decoding
with greedy acceptance reproduces plain greedy decoding token for token.
"""
import math
import os
import re

import numpy as np
import pytest

import oracle
import respec_synth as synth
from oracle import draft as od

import decode_loop as dl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _trigger_cases():
    out = []
    for line in open(os.path.join(GOLDEN, "trigger_cases.txt")):
        line = line.split("#")[0].strip()
        if not line:
            continue
        f = line.split()
        ent = [float(x) for x in f[0].split(",")]
        out.append((ent, int(f[1]), float(f[2]), float(f[3]), int(f[4]), float(f[5]), float(f[6]), int(f[7])))
    return out


@pytest.mark.parametrize("case", _trigger_cases(), ids=lambda c: ",".join(map(str, c[0])))
def test_trigger_hand_worked(case):
    ent, l, lam, theta, k_exp, h_exp, c_exp, fire_exp = case
    k, h, c, fire = od.trigger_eval(ent, l, lam, theta)
    assert k == k_exp
    assert int(fire) == fire_exp
    if k_exp == 0:
        assert math.isnan(h) and math.isnan(c)
    else:
        assert h == pytest.approx(h_exp, abs=1e-12)
        assert c == pytest.approx(c_exp, abs=1e-12)


def test_trigger_constant_entropy_closed_form():
    # H_k = e for every k, so C_k = e + lambda/k: the longest key wins for
    # lambda > 0, the shortest for lambda < 0, and the smallest k on the tie at 0
    rng = np.random.default_rng(1)
    for _ in range(50):
        e = float(rng.uniform(0, 5))
        n, l = int(rng.integers(1, 8)), int(rng.integers(1, 6))
        lam = float(rng.uniform(0.01, 2))
        k, h, c, _ = od.trigger_eval([e] * n, l, lam, 1.5)
        assert k == min(l, n) and h == pytest.approx(e) and c == pytest.approx(e + lam / k)
        assert od.trigger_eval([e] * n, l, -lam, 1.5)[0] == 1
        assert od.trigger_eval([e] * n, l, 0.0, 1.5)[0] == 1


def test_trigger_lambda_zero_is_the_least_suffix_mean():
    # with lambda = 0, k* is the first minimum of the suffix means, computed
    # here with numpy's cumulative sum over the reversed window
    rng = np.random.default_rng(2)
    for _ in range(200):
        n = int(rng.integers(1, 9))
        l = int(rng.integers(1, 9))
        ent = rng.choice([0.25, 0.5, 1.0, 2.0, 3.0], size=n)   # ties are common
        means = np.cumsum(ent[::-1])[:min(l, n)] / np.arange(1, min(l, n) + 1)
        k, h, _, fire = od.trigger_eval(list(ent), l, 0.0, 1.0)
        assert k == int(np.argmin(means)) + 1
        assert h == pytest.approx(float(means.min()))
        assert fire == (means.min() <= 1.0)


def _regex_positions(text, key):
    # every end index of an occurrence, found with a zero-width look-ahead
    s = "".join(chr(65 + t) for t in text)
    k = "".join(chr(65 + t) for t in key)
    ends = [m.start() + len(key) - 1 for m in re.finditer(f"(?=({re.escape(k)}))", s)]
    return sorted([p for p in ends if p < len(text) - 1], reverse=True)


def test_positions_hand_worked():
    text = [5, 6, 7, 5, 6, 7, 5, 6]
    assert od.positions(text, [5, 6]) == [4, 1]       # the trailing occurrence has no continuation
    assert od.positions(text, [7]) == [5, 2]
    assert od.positions(text, [6, 7, 5]) == [6, 3]
    assert od.positions(text, [7, 5, 6]) == [4]
    assert od.positions(text, [8]) == []
    assert od.positions(text, text) == []


def test_positions_against_a_regex_scan():
    rng = np.random.default_rng(3)
    for _ in range(300):
        n = int(rng.integers(1, 60))
        a = int(rng.integers(1, 5))
        text = [int(x) for x in rng.integers(0, a, n)]
        k = int(rng.integers(1, 5))
        key = text[n - k:] if (rng.random() < 0.5 and k <= n) else [int(x) for x in rng.integers(0, a, k)]
        assert od.positions(text, key) == _regex_positions(text, key)


def test_ema_closed_form():
    # n updates with a constant rate R from S_0: S_n = R + (S_0 - R)(1 - alpha)^n
    for alpha in (0.25, 0.5, 0.9):
        for l_acc, l_draft in ((0, 4), (3, 4), (5, 5)):
            sc = {}
            for _ in range(7):
                od.ema_update(sc, [10], 0, l_acc, [l_draft], alpha, 0.5)
            r = l_acc / l_draft
            assert sc[10] == pytest.approx(r + (0.5 - r) * (1 - alpha) ** 7, abs=1e-12)


def test_ema_and_selection_hand_worked():
    sc = {}
    # winner gets R = 2/4; the other selected position R = 0 (Algorithm 1's feedback)
    od.ema_update(sc, [7, 3], 0, 2, [4, 4], 0.5, 0.5)
    assert sc == {7: 0.5, 3: 0.25}
    # threshold 0.3 drops position 3; unseen positions 9 and 1 score s0 = 0.5 and tie
    # with 7, the more recent first
    assert od.select(sc, [9, 7, 3, 1], 0.5, 0.3, 0.5, 3) == [9, 7, 1]
    assert od.select(sc, [9, 7, 3, 1], 0.5, 0.3, 0.5, 2) == [9, 7]
    assert od.select(sc, [3], 0.5, 0.3, 0.5, 3) == []


def test_build_tree_hand_worked():
    text = [9, 1, 2, 3, 9, 1, 2, 4, 9, 1, 5, 9]
    sel = od.positions(text, [9])
    assert sel == [8, 4, 0]
    parent, token, src, ce, cl = od.build_tree(text, sel, 3, 61)
    assert parent == [-1, 0, 1, 2, 1, 4, 4]
    assert token == [9, 1, 5, 9, 2, 4, 3]
    assert src == [0, 1, 1, 1, 1, 1, 1]
    assert ce == [3, 5, 6] and cl == [3, 3, 3]
    # a budget of 5 nodes cuts the second and third continuations after "1 2"
    parent, token, src, ce, cl = od.build_tree(text, sel, 3, 5)
    assert parent == [-1, 0, 1, 2, 1] and token == [9, 1, 5, 9, 2]
    assert ce == [3, 4, 4] and cl == [3, 2, 2]


def test_build_tree_is_the_trie_of_the_continuations():
    rng = np.random.default_rng(4)
    for _ in range(200):
        n = int(rng.integers(2, 80))
        text = [int(x) for x in rng.integers(0, 3, n)]
        sel = sorted(set(int(x) for x in rng.integers(0, n - 1, int(rng.integers(1, 6)))), reverse=True)
        dlen = int(rng.integers(1, 12))
        parent, token, src, ce, cl = od.build_tree(text, sel, dlen, 10 ** 6)
        conts = [tuple(text[p + 1: p + 1 + dlen]) for p in sel]
        prefixes = {c[:i] for c in conts for i in range(1, len(c) + 1)}
        assert len(parent) == 1 + len(prefixes)                  # one node per distinct prefix
        assert all(0 <= parent[j] < j for j in range(1, len(parent)))

        def spell(v):
            out = []
            while v > 0:
                out.append(token[v])
                v = parent[v]
            return tuple(reversed(out))
        assert {spell(v) for v in range(1, len(parent))} == prefixes
        for c, end, ln in zip(conts, ce, cl):
            assert spell(end) == c and ln == len(c)
        # sibling tokens are distinct (a trie)
        seen = set()
        for j in range(1, len(parent)):
            assert (parent[j], token[j]) not in seen
            seen.add((parent[j], token[j]))


class _OracleSession:
    def __init__(self, **kw):
        self.s = od.Session(**kw)

    def append(self, t, e):
        self.s.append([int(x) for x in t], e)

    def propose(self):
        r = self.s.propose()
        return r["parent"], r["token"], r["src"], r["retrieved"]

    def commit(self, *a):
        self.s.commit(*a)

    def text(self):
        return list(self.s.text)


def test_strict_speculative_decoding_equals_greedy_decoding():
    # Algorithm 1 with greedy strict verification (k = 1: only the argmax
    # passes) is lossless: whatever the retrieval drafts, the generated text is
    # the one plain greedy decoding produces
    m = dl.make_model(params=synth.AcceptParams(topk=1, tau=0.0, min_lookahead=2, max_relaxed=2))
    pr = dl.prompt()
    text, steps = dl.speculative_decode(m, _OracleSession(), pr, 60, oracle.verify_step)
    assert sum(r for r, _, _ in steps) >= 3 and max(a for _, _, a in steps) >= 3   # retrieval did draft
    ar = dl.greedy_decode(m, pr, len(text) - len(pr), oracle.verify_step)
    assert text == ar


def test_relaxed_loop_accepts_more_and_keeps_its_invariants():
    # with relaxed verification the loop accepts at least as many tokens per
    # retrieval step on this workload, and every committed step appends
    # acc_len + 1 tokens
    m = dl.make_model(params=synth.AcceptParams(topk=8, tau=3.0, min_lookahead=2, max_relaxed=2))
    pr = dl.prompt()
    s = _OracleSession()
    text, steps = dl.speculative_decode(m, s, pr, 40, oracle.verify_step)
    assert len(text) == len(pr) + sum(a + 1 for _, _, a in steps)
    assert max(a for _, _, a in steps) >= 10
    assert all(n == 1 for r, n, _ in steps if not r)
