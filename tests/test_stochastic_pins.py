"""Pins of the oracle's stochastic (lossless) verification.

Section 3.4 verifies drafter outputs with standard lossless speculative
sampling.  What fixes it, independently of the oracle's code: hand-worked
acceptance probabilities and residual draws; the defining property that the
emitted token is distributed exactly as the target distribution whatever the
drafts (checked by Monte Carlo over the input uniforms, for several siblings
mixing model-drafted and retrieved drafts); a drafter equal to the target
accepts every draft; and at a vanishing temperature the procedure reduces to
greedy strict verification.
"""
import math

import numpy as np
import pytest

import oracle


def _log(p):
    return np.log(np.asarray(p, np.float64)).astype(np.float32)


def test_hand_worked_deterministic_draft():
    # p = (.1, .2, .3, .4); a retrieved (one-hot) draft of token 3 is accepted
    # with probability p(3) = 0.4; after its rejection the residual is p with
    # token 3 removed, (1/6, 2/6, 3/6, 0), and u = 0.4 draws token 1
    z = _log([0.1, 0.2, 0.3, 0.4])
    assert oracle.stoch_node(z, 1.0, None, [3], [0], [0.4 - 1e-6], 0.4) == (0, -1)
    assert oracle.stoch_node(z, 1.0, None, [3], [0], [0.4 + 1e-6], 0.4) == (-1, 1)
    assert oracle.stoch_node(z, 1.0, None, [3], [0], [0.9], 0.5 - 1e-6) == (-1, 1)
    assert oracle.stoch_node(z, 1.0, None, [3], [0], [0.9], 0.5 + 1e-6) == (-1, 2)
    # a leaf draws from p itself: cumulative (.1, .3, .6, 1)
    assert oracle.stoch_node(z, 1.0, None, [], [], [], 0.05)[1] == 0
    assert oracle.stoch_node(z, 1.0, None, [], [], [], 0.65)[1] == 3


def test_hand_worked_model_draft():
    # q = (.4, .3, .2, .1) drafted token 0: accept with min(1, .1/.4) = 0.25;
    # the residual max(p - q, 0) = (0, 0, .1, .3) normalises to (0, 0, .25, .75)
    z = _log([0.1, 0.2, 0.3, 0.4])
    q = np.array([0.4, 0.3, 0.2, 0.1], np.float32)
    assert oracle.stoch_node(z, 1.0, q, [0], [1], [0.25 - 1e-6], 0.0) == (0, -1)
    assert oracle.stoch_node(z, 1.0, q, [0], [1], [0.25 + 1e-6], 0.2) == (-1, 2)
    assert oracle.stoch_node(z, 1.0, q, [0], [1], [0.5], 0.3) == (-1, 3)
    # drafted token 3 (q = .1 < p = .4) is always accepted
    assert oracle.stoch_node(z, 1.0, q, [3], [1], [0.999], 0.5) == (0, -1)
    # temperature: p = softmax(z / 2) = normalised sqrt(p)
    s = np.sqrt([0.1, 0.2, 0.3, 0.4])
    p2 = s / s.sum()
    assert oracle.stoch_node(z, 2.0, None, [3], [0], [p2[3] - 1e-6], 0.5) == (0, -1)
    assert oracle.stoch_node(z, 2.0, None, [3], [0], [p2[3] + 1e-6], 0.5)[0] == -1


@pytest.mark.parametrize("kinds", ["m", "r", "mm", "mr", "rmr", "mmm"])
def test_emitted_token_is_distributed_as_the_target(kinds):
    # Monte Carlo over the uniforms and the drafts: model drafts are sampled
    # from q, retrieved drafts are fixed tokens; the emitted token (the first
    # accepted draft, or the residual draw) must follow p whatever the drafts
    rng = np.random.default_rng(sum(map(ord, kinds)))
    V, N = 6, 40000
    z = rng.normal(0, 1.0, V).astype(np.float32)
    T = 0.8
    p = np.exp(z.astype(np.float64) / T)
    p /= p.sum()
    q = rng.dirichlet(np.ones(V)).astype(np.float32)
    qd = q.astype(np.float64) / q.astype(np.float64).sum()
    fixed = [int(rng.integers(0, V)) for _ in kinds]
    counts = np.zeros(V)
    for _ in range(N):
        toks = [int(rng.choice(V, p=qd)) if k == "m" else fixed[i] for i, k in enumerate(kinds)]
        u = rng.random(len(kinds) + 1).astype(np.float32)
        k, s = oracle.stoch_node(z, T, q, toks, [c == "m" for c in kinds], u[:-1], float(u[-1]))
        counts[toks[k] if k >= 0 else s] += 1
    freq = counts / N
    sigma = np.sqrt(p * (1 - p) / N)
    assert np.all(np.abs(freq - p) <= 5 * sigma + 1e-4), (freq, p)


def test_drafter_equal_to_target_accepts_every_draft():
    rng = np.random.default_rng(7)
    for _ in range(50):
        V = int(rng.integers(2, 50))
        z = rng.normal(0, 2, V).astype(np.float32)
        T = float(rng.uniform(0.5, 2))
        p = np.exp((z.astype(np.float64) - z.max()) / T)
        q = (p / p.sum()).astype(np.float32)
        t = int(rng.integers(0, V))
        # a = min(1, p(t)/q(t)) = 1 up to float32 rounding of q
        k, _ = oracle.stoch_node(z, T, q, [t, (t + 1) % V], [1, 1], [0.999, 0.999], 0.5)
        pt = float(p[t] / p.sum())
        assert k == 0 or pt / float(q[t]) < 0.999


def _greedy_walk(parent, token, z):
    n = len(parent)
    cur, path = 0, [0]
    while True:
        nxt = [j for j in range(1, n) if parent[j] == cur and token[j] == int(np.argmax(z[cur]))]
        if not nxt:
            return path, int(np.argmax(z[cur]))
        cur = nxt[0]
        path.append(cur)


def test_vanishing_temperature_is_greedy_strict_verification():
    # logits with top-1 gaps >= 0.5 at T = 1e-3: p is one-hot to double
    # precision, so every draft is accepted iff it is the parent's argmax and
    # the residual draw is the argmax: the walk is greedy verification
    rng = np.random.default_rng(8)
    for trial in range(40):
        n, V = int(rng.integers(2, 20)), 50
        parent = [-1] + [int(rng.integers(0, j)) for j in range(1, n)]
        z = rng.normal(0, 1, (n, V))
        am = rng.integers(0, V, n)
        for i in range(n):
            z[i, am[i]] = z[i].max() + 0.5 + rng.random()
        z = z.astype(np.float32)
        token = [0] * n
        for j in range(1, n):     # distinct sibling tokens; about half are the argmax
            sib = [token[k] for k in range(1, j) if parent[k] == parent[j]]
            cand = int(am[parent[j]]) if (rng.random() < 0.6 and int(am[parent[j]]) not in sib) else None
            while cand is None or cand in sib:
                cand = int(rng.integers(0, V))
            token[j] = cand
        src = [0] + [int(rng.integers(0, 2)) for _ in range(1, n)]
        q = rng.dirichlet(np.ones(V), n).astype(np.float32)
        u = rng.uniform(0.01, 0.99, (n, 2)).astype(np.float32)
        out = oracle.stochastic(parent, token, src, z, q, u, 1e-3, 32)
        path, bonus = _greedy_walk(parent, token, z)
        assert out["path"][:len(path)].tolist() == path and out["acc_len"] == len(path) - 1
        assert out["bonus"] == bonus


def test_walk_invariants():
    rng = np.random.default_rng(9)
    for trial in range(60):
        n, V = int(rng.integers(1, 30)), 40
        parent = [-1] + [int(rng.integers(max(0, j - 4), j)) for j in range(1, n)]
        token = [0] + [int(rng.integers(0, V)) for _ in range(1, n)]
        src = [0] + [int(rng.integers(0, 2)) for _ in range(1, n)]
        z = rng.normal(0, 1.5, (n, V)).astype(np.float32)
        q = rng.dirichlet(np.ones(V) * 0.3, n).astype(np.float32)
        u = rng.random((n, 2)).astype(np.float32)
        out = oracle.stochastic(parent, token, src, z, q, u, 1.0, 32)
        acc = out["acc_len"]
        path = out["path"][:acc + 1].tolist()
        assert path[0] == 0 and all(parent[path[d]] == path[d - 1] for d in range(1, acc + 1))
        assert all(x == -1 for x in out["path"][acc + 1:])
        # the walk follows the first accepted child; it stops where none is
        for d in range(acc):
            assert out["first_acc"][path[d]] == path[d + 1]
        assert out["first_acc"][path[-1]] == -1 and out["bonus"] == out["sample"][path[-1]] >= 0
        # acc_bit marks exactly the first accepted children, which are the
        # earliest children of their parents that pass
        for j in range(1, n):
            assert out["acc_bit"][j] == (out["first_acc"][parent[j]] == j)
        is_leaf = [all(parent[k] != i for k in range(n)) for i in range(n)]
        for l in range(n):
            if not is_leaf[l]:
                assert out["leaf_acc_len"][l] == -1
                continue
            chain, v = [], l
            while v > 0:
                chain.append(v)
                v = parent[v]
            assert out["leaf_acc_len"][l] == len(set(chain) & set(path))
        wl = out["winner_leaf"]
        assert is_leaf[wl]
        v = wl
        while v != path[-1] and v > 0:
            v = parent[v]
        assert v == path[-1]
