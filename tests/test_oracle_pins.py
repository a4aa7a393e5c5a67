"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: a library
routine (torch SDPA in float64, numpy matmul, scipy entropy/logsumexp, a
stable sort), a closed form, an invariant, a hand-worked case from the paper's
prose, or brute force on tiny inputs.
"""
import itertools
import math
import os

import numpy as np
import pytest
import torch
from scipy import special, stats

import oracle
import respec_synth as synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _shape(dtype="bf16", hd=128, hq=2, hkv=1, d=64, v=512, b=1, n=16, depth=8, topk_out=8):
    return synth.Shape("pin", dtype, hd, hq, hkv, d, v, b, n, depth, topk_out)


def _ancestors_by_closure(parent):
    """Ancestor-or-self matrix via boolean matrix powers (not a parent walk)."""
    n = len(parent)
    A = np.zeros((n, n), dtype=np.int64)
    for j in range(1, n):
        A[j, parent[j]] = 1
    R = np.eye(n, dtype=np.int64)
    P = np.eye(n, dtype=np.int64)
    for _ in range(n):
        P = np.minimum(P @ A, 1)
        R = np.minimum(R + P, 1)
    return R.astype(np.uint8)


def _to_f64(w, arr):
    if w.shape.dtype == "bf16":
        return synth.bf16_bits_to_f32(arr).astype(np.float64)
    return np.asarray(arr, dtype=np.float64)


def _sdpa_reference(w, b, mask_tree):
    """torch SDPA (float64, CPU) over [prefix ++ tree rows] with a boolean mask."""
    shp = w.shape
    lo, hi = int(w.node_off[b]), int(w.node_off[b + 1])
    n, L = hi - lo, int(w.kv_len[b])
    G = shp.n_q_heads // shp.n_kv_heads
    q = torch.from_numpy(_to_f64(w, w.hidden[lo:hi])).view(n, shp.n_q_heads, shp.head_dim)
    q = q.permute(1, 0, 2).unsqueeze(0)                       # [1, Hq, n, D]
    k = torch.from_numpy(_to_f64(w, w.k_cache[b][:, :L + n]))  # [Hkv, L+n, D]
    v = torch.from_numpy(_to_f64(w, w.v_cache[b][:, :L + n]))
    k = k.repeat_interleave(G, dim=0).unsqueeze(0)
    v = v.repeat_interleave(G, dim=0).unsqueeze(0)
    mask = torch.zeros(n, L + n, dtype=torch.bool)
    mask[:, :L] = True
    mask[:, L:] = torch.from_numpy(mask_tree.astype(bool))
    o = torch.nn.functional.scaled_dot_product_attention(q, k, v, attn_mask=mask)
    return o.squeeze(0).permute(1, 0, 2).reshape(n, shp.n_q_heads * shp.head_dim).numpy()


def _oracle_attn(w, b):
    shp = w.shape
    lo, hi = int(w.node_off[b]), int(w.node_off[b + 1])
    st, depth, anc, leaf = oracle.tree(w.parent[lo:hi], shp.max_depth)
    assert st == 0
    dt = oracle.BF16 if shp.dtype == "bf16" else oracle.F32
    return oracle.attention(dt, w.hidden[lo:hi], w.k_cache[b], w.v_cache[b], int(w.kv_len[b]), anc,
                            shp.n_q_heads, shp.n_kv_heads, shp.head_dim)


# ---------------------------------------------------------------------------
# tree
# ---------------------------------------------------------------------------

def test_tree_matches_closure_on_all_small_trees():
    for n in range(1, 7):
        for choice in itertools.product(*[range(j) for j in range(1, n)]):
            parent = [-1] + list(choice)
            st, depth, anc, leaf = oracle.tree(parent, 16)
            assert st == 0
            ref = _ancestors_by_closure(parent)
            assert np.array_equal(anc[:n, :n], ref)
            assert np.array_equal(depth[:n], ref.sum(axis=1) - 1)
            has_child = np.zeros(n, bool)
            for j in range(1, n):
                has_child[parent[j]] = True
            assert np.array_equal(leaf[:n].astype(bool), ~has_child)


@pytest.mark.parametrize("parent,max_depth,code", [
    ([0, 0], 4, 1),            # root must have parent -1
    ([-1, 1], 4, 2),           # self parent
    ([-1, 0, 3, 1], 4, 2),     # forward reference
    ([-1, -1], 4, 2),          # second root
    ([-1, 0, 1, 2], 2, 3),     # depth 3 > max 2
])
def test_tree_rejects_malformed(parent, max_depth, code):
    st, *_ = oracle.tree(parent, max_depth)
    assert st == code


# ---------------------------------------------------------------------------
# attention
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("dtype,hq,hkv", [("bf16", 4, 4), ("bf16", 4, 2), ("f32", 2, 1)])
def test_chain_tree_equals_causal_attention(dtype, hq, hkv):
    n, L = 7, 37
    shp = _shape(dtype, hd=hq * 32, hq=hq, hkv=hkv, d=32)
    w = synth.custom(shp, [[-1] + list(range(n - 1))], [L], seed=11)
    causal = np.tril(np.ones((n, n), dtype=np.uint8))  # textbook causal mask on the new rows
    ref = _sdpa_reference(w, 0, causal)
    np.testing.assert_allclose(_oracle_attn(w, 0), ref, rtol=1e-12, atol=1e-12)


def test_single_node_equals_decode_attention():
    shp = _shape("bf16", hd=128, hq=4, hkv=2, d=32)
    w = synth.custom(shp, [[-1]], [50], seed=12)
    ref = _sdpa_reference(w, 0, np.ones((1, 1), np.uint8))
    np.testing.assert_allclose(_oracle_attn(w, 0), ref, rtol=1e-12, atol=1e-12)


def test_star_tree_sees_prefix_root_and_self():
    n = 6
    shp = _shape("bf16", hd=64, hq=2, hkv=2, d=32)
    w = synth.custom(shp, [[-1] + [0] * (n - 1)], [20], seed=13)
    mask = np.eye(n, dtype=np.uint8)
    mask[:, 0] = 1
    ref = _sdpa_reference(w, 0, mask)
    np.testing.assert_allclose(_oracle_attn(w, 0), ref, rtol=1e-12, atol=1e-12)


def test_random_tree_and_empty_prefix_match_masked_sdpa():
    shp = _shape("bf16", hd=128, hq=4, hkv=1, d=32)
    parents = [[-1, 0, 0, 1, 1, 2, 5, 6, 3], [-1, 0, 1, 0]]
    w = synth.custom(shp, parents, [9, 0], seed=14)
    for b in range(2):
        ref = _sdpa_reference(w, b, _ancestors_by_closure(parents[b]))
        np.testing.assert_allclose(_oracle_attn(w, b), ref, rtol=1e-12, atol=1e-12)


def test_gqa_equals_mha_with_replicated_heads():
    shp = _shape("bf16", hd=128, hq=4, hkv=1, d=32)
    w = synth.custom(shp, [[-1, 0, 1, 0]], [15], seed=15)
    shp2 = _shape("bf16", hd=128, hq=4, hkv=4, d=32)
    w2 = synth.custom(shp2, [[-1, 0, 1, 0]], [15], seed=15)
    w2.hidden = w.hidden
    w2.k_cache = np.repeat(w.k_cache, 4, axis=1)
    w2.v_cache = np.repeat(w.v_cache, 4, axis=1)
    np.testing.assert_array_equal(_oracle_attn(w, 0), _oracle_attn(w2, 0))


# ---------------------------------------------------------------------------
# residual, logits
# ---------------------------------------------------------------------------

def _nearest_bf16(d: float) -> float:
    """Brute force: the bf16 value nearest to d, ties to the even bit pattern."""
    b0 = int(np.array([d], np.float32).view(np.uint32)[0]) >> 16
    cands = [b for b in range(b0 - 2, b0 + 3) if 0 <= b < 0x10000]
    vals = [(abs(float(np.array([b << 16], np.uint32).view(np.float32)[0]) - d), b & 1, b) for b in cands]
    best = min(vals)
    return float(np.array([best[2] << 16], np.uint32).view(np.float32)[0])


def test_residual_rounds_the_exact_sum_once_to_bf16():
    # x = RNE_bf16(h + O) of the exact (double) sum.  Besides random sums: exact
    # midpoints between neighbouring bf16 values (ties go to the even pattern) and
    # sums a hair above or below a midpoint, which a float32 sum would first round
    # onto the midpoint (rounding twice then goes the wrong way on half of them).
    rng = np.random.default_rng(0)
    hb = synth.f32_to_bf16_bits(rng.standard_normal(4096).astype(np.float32))
    h = synth.bf16_bits_to_f32(hb).astype(np.float64)
    o = rng.standard_normal(4096) * 0.05
    up = (hb.astype(np.uint32) + 1).astype(np.uint16)
    mid = (h + synth.bf16_bits_to_f32(up).astype(np.float64)) / 2
    o[:1024] = mid[:1024] - h[:1024]                          # exact ties
    o[1024:2048] = mid[1024:2048] - h[1024:2048] + np.abs(h[1024:2048]) * 2.0 ** -40
    o[2048:3072] = mid[2048:3072] - h[2048:3072] - np.abs(h[2048:3072]) * 2.0 ** -40
    x = oracle.residual(oracle.BF16, hb, o)
    ref = np.array([_nearest_bf16(float(a) + float(b)) for a, b in zip(h, o)])
    np.testing.assert_array_equal(x, ref)
    # and in float32 workloads, numpy's round-to-nearest-even cast of the double sum
    hf = rng.standard_normal(4096).astype(np.float32)
    x32 = oracle.residual(oracle.F32, hf, o)
    np.testing.assert_array_equal(x32, (hf.astype(np.float64) + o).astype(np.float32).astype(np.float64))


def test_logits_match_library_gemm():
    rng = np.random.default_rng(1)
    x = synth.bf16_bits_to_f32(synth.f32_to_bf16_bits(rng.standard_normal((5, 96)).astype(np.float32)))
    W = synth.f32_to_bf16_bits((rng.standard_normal((77, 96)) * 0.02).astype(np.float32))
    z = oracle.logits(oracle.BF16, x.astype(np.float64), W)
    ref = x.astype(np.float64) @ synth.bf16_bits_to_f32(W).astype(np.float64).T
    np.testing.assert_allclose(z, ref, rtol=1e-13, atol=1e-13)


# ---------------------------------------------------------------------------
# row statistics (Eq. 1 entropy, log-softmax, top-k)
# ---------------------------------------------------------------------------

def test_row_stats_match_scipy_and_stable_sort():
    rng = np.random.default_rng(2)
    z = (rng.standard_normal((6, 1000)) * 1.3).astype(np.float32)
    z[3, 10] = z[3, 20] = z[3].max() + 1.0      # tied maximum: smallest id wins
    z[4, 100:110] = 2.5                          # ties inside the top-k
    st = oracle.row_stats(z, 8)
    zd = z.astype(np.float64)
    np.testing.assert_allclose(st["lse"], special.logsumexp(zd, axis=1), rtol=1e-13)
    np.testing.assert_allclose(st["entropy"], stats.entropy(special.softmax(zd, axis=1), axis=1),
                               rtol=1e-11)
    np.testing.assert_array_equal(st["argmax"], np.argmax(z, axis=1))
    np.testing.assert_array_equal(st["max_logit"], zd.max(axis=1))
    for r in range(6):
        order = np.lexsort((np.arange(1000), -zd[r]))
        np.testing.assert_array_equal(st["topk_id"][r], order[:8])
        np.testing.assert_allclose(st["topk_logprob"][r], zd[r, order[:8]] - st["lse"][r], rtol=1e-13)
        for t in (0, 5, int(order[3]), int(order[500])):
            assert oracle.rank(z[r], t) == int(np.nonzero(order == t)[0][0])
    assert st["argmax"][3] == 10


@pytest.mark.parametrize("vocab", [4096, 32000, 128256])
def test_uniform_row_has_entropy_log_v(vocab):
    # W = 0 gives z = 0: p is uniform, H = lse = log V, argmax = 0 (tie rule)
    st = oracle.row_stats(np.zeros((1, vocab), np.float32), 4)
    assert abs(st["entropy"][0] - math.log(vocab)) < 1e-9
    assert abs(st["lse"][0] - math.log(vocab)) < 1e-12
    assert st["argmax"][0] == 0
    np.testing.assert_array_equal(st["topk_id"][0], [0, 1, 2, 3])


def test_dominant_logit_entropy_closed_form():
    V = 1000
    z = np.zeros((1, V), np.float32)
    z[0, 7] = 30.0
    st = oracle.row_stats(z, 2)
    S = math.exp(30.0) + (V - 1)
    p1, p = math.exp(30.0) / S, 1.0 / S
    H = -(p1 * math.log(p1) + (V - 1) * p * math.log(p))
    assert abs(st["entropy"][0] - H) < 1e-12
    assert st["entropy"][0] < 1e-8
    assert st["argmax"][0] == 7


# ---------------------------------------------------------------------------
# acceptance predicates (Section 3.4, Eq. 6-7) and look-ahead tolerance
# ---------------------------------------------------------------------------

def test_node_flags_hand_built_row():
    V = 10
    z = np.zeros((2, V), np.float32)
    z[0] = [0.0, 5.0, 4.0, 3.5, 1.0, 4.0, -1.0, 0.5, 2.0, 1.9]   # argmax 1; order 1,2,5,3,8,9,4,7,0,6
    parent = [-1, 0, 0, 0, 0, 0]
    token = [0, 1, 5, 3, 8, 6]
    src = [0, 1, 1, 1, 0, 1]
    st = oracle.row_stats(z, 4)
    flags, lp, rk = oracle.node_flags(parent, token, src, np.vstack([z[0]] * 6), np.full(6, st["argmax"][0]),
                                      np.full(6, st["lse"][0]), topk=3, tau=1.6)
    # rank: token1 -> 0, token5 -> 2 (ties with 2 broken by id), token3 -> 3, token8 -> 4, token6 -> 9
    np.testing.assert_array_equal(rk, [-1, 0, 2, 3, 4, 9])
    G, T, U, R = oracle.FLAG_GREEDY, oracle.FLAG_TOPK, oracle.FLAG_TAU, oracle.FLAG_RELAXED
    np.testing.assert_array_equal(flags, [0, G | T | U | R, T | U | R, U, 0, 0])
    np.testing.assert_allclose(lp[1:], z[0, token[1:]] - st["lse"][0])


def _golden_cases():
    cases = []
    with open(os.path.join(GOLDEN, "lookahead_cases.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            pat, m, phi, exp = line.split()
            cases.append(("" if pat == "-" else pat, int(m), int(phi), int(exp)))
    return cases


def _pattern_arrays(pat):
    g = np.array([c == "G" for c in pat], np.uint8)
    ok = np.array([c in "GR" for c in pat], np.uint8)
    return g, ok


@pytest.mark.parametrize("pat,m,phi,expected", _golden_cases())
def test_lookahead_hand_worked_cases(pat, m, phi, expected):
    g, ok = _pattern_arrays(pat)
    assert oracle.lookahead(g, ok, m, phi) == expected


def test_lookahead_invariants_on_all_short_patterns():
    for d in range(0, 8):
        for pat in itertools.product("GRX", repeat=d):
            pat = "".join(pat)
            g, ok = _pattern_arrays(pat)
            l0 = next((i for i, c in enumerate(pat) if c != "G"), d)
            for m in range(0, 4):
                for phi in range(0, 4):
                    acc = oracle.lookahead(g, ok, m, phi)
                    acc_path = pat[:acc]
                    assert l0 <= acc <= d
                    if phi == 0:
                        assert acc == l0                     # no relaxed attempt: strict greedy
                    assert "X" not in acc_path               # every accepted node passes
                    non_greedy = [i for i, c in enumerate(acc_path) if c != "G"]
                    assert len(non_greedy) <= phi            # at most Phi relaxed tokens
                    if non_greedy:                           # the last one has >= m greedy after it
                        tail = acc_path[non_greedy[-1] + 1:]
                        assert len(tail) >= m and set(tail) <= {"G"}
                        # and the run is maximal: acceptance stops at a non-greedy node or the end
                        assert acc == d or pat[acc] != "G"
                    if "X" not in pat and "R" not in pat:
                        assert acc == d


def test_lookahead_fully_lenient_accepts_whole_chain():
    # tau = inf, k = V, m = 0, Phi >= d on an all-retrieved chain: everything passes
    for d in range(0, 9):
        for pat in itertools.product("GR", repeat=d):
            g, ok = _pattern_arrays("".join(pat))
            assert oracle.lookahead(g, ok, 0, d) == d


def _brute_force_path(parent, flags, argmax, m, phi):
    n = len(parent)
    children = [[] for _ in range(n)]
    for j in range(1, n):
        children[parent[j]].append(j)
    chains = []

    def dfs(node, chain):
        if not children[node]:
            chains.append(list(chain))
            return
        for c in children[node]:
            dfs(c, chain + [c])

    dfs(0, [])
    leaf_acc = np.full(n, -1, np.int32)
    cands = []
    for ch in chains:
        leaf = ch[-1] if ch else 0
        g = np.array([(flags[u] & oracle.FLAG_GREEDY) != 0 for u in ch], np.uint8)
        ok = np.array([(flags[u] & (oracle.FLAG_GREEDY | oracle.FLAG_RELAXED)) != 0 for u in ch], np.uint8)
        acc = oracle.lookahead(g, ok, m, phi)
        leaf_acc[leaf] = acc
        accepted = [0] + ch[:acc]
        cands.append((-acc, accepted[-1], leaf, accepted))
    best = min(cands)
    return leaf_acc, -best[0], best[3], best[2], argmax[best[1]]


def test_tree_winner_matches_brute_force_enumeration():
    rng = np.random.default_rng(3)
    for n in range(1, 7):
        for choice in itertools.product(*[range(j) for j in range(1, n)]):
            parent = [-1] + list(choice)
            st, depth, anc, leaf = oracle.tree(parent, 8)
            for trial in range(3):
                flags = np.zeros(n, np.uint8)
                kinds = rng.integers(0, 3, n)
                for j in range(1, n):
                    flags[j] = {0: oracle.FLAG_GREEDY | oracle.FLAG_RELAXED, 1: oracle.FLAG_RELAXED, 2: 0}[kinds[j]]
                argmax = rng.integers(0, 100, n).astype(np.int32)
                m, phi = int(rng.integers(0, 3)), int(rng.integers(0, 3))
                f = flags.copy()
                res = oracle.path(parent, leaf, depth, f, argmax, 8, m, phi)
                leaf_acc, acc, accepted, wl, bonus = _brute_force_path(parent, flags, argmax, m, phi)
                np.testing.assert_array_equal(res["leaf_acc_len"], leaf_acc)
                assert res["acc_len"] == acc
                assert res["path"][:acc + 1].tolist() == accepted
                assert (res["path"][acc + 1:] == -1).all()
                assert res["winner_leaf"] == wl
                assert res["bonus"] == bonus
                on = np.nonzero(f & oracle.FLAG_ON_PATH)[0].tolist()
                assert on == sorted(accepted)


# ---------------------------------------------------------------------------
# whole step: strict / relaxed special cases
# ---------------------------------------------------------------------------

def _greedy_walk_case(dtype, seed):
    shp = _shape(dtype, hd=128, hq=4, hkv=2, d=32, v=600, n=9, depth=8)
    parent = [-1, 0, 1, 2, 3, 4, 5, 6, 7]
    w = synth.custom(shp, [parent], [33], seed=seed)
    f = oracle.forward(w)
    am = np.argmax(f["z"].astype(np.float32), axis=1)
    return w, f, am


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_strict_chain_of_greedy_tokens_accepts_whole_depth(dtype):
    w, f, am = _greedy_walk_case(dtype, 21)
    w.token = np.array([w.token[0]] + [am[j - 1] for j in range(1, 9)], np.int32)
    w.src[:] = synth.SRC_MODEL
    d = oracle.decide(w, f["z"])
    assert d["acc_len"][0] == 8
    assert d["path"][0].tolist() == list(range(9))
    assert d["bonus"][0] == am[8]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_strict_all_model_tree_reproduces_greedy_decoding(dtype):
    # a tree whose every branch point offers the greedy token among others
    shp = _shape(dtype, hd=128, hq=4, hkv=2, d=32, v=600, n=13, depth=8)
    parent = [-1, 0, 0, 1, 1, 3, 3, 5, 5, 7, 7, 9, 9]
    w = synth.custom(shp, [parent], [40], seed=22)
    w.src[:] = synth.SRC_MODEL
    f = oracle.forward(w)
    am = np.argmax(f["z"].astype(np.float32), axis=1)
    tok = w.token.copy()
    for j in range(1, 13):
        if j % 2 == 1:
            tok[j] = am[parent[j]]
        elif tok[j] == am[parent[j]]:
            tok[j] = (tok[j] + 1) % 600
    w.token = tok
    d = oracle.decide(w, f["z"])
    # greedy decoding from the root: follow argmax while the tree holds it
    walk, node = [0], 0
    while True:
        nxt = [c for c in range(1, 13) if parent[c] == node and tok[c] == am[node]]
        if not nxt:
            break
        node = nxt[0]
        walk.append(node)
    assert d["path"][0][:len(walk)].tolist() == walk
    assert d["acc_len"][0] == len(walk) - 1
    assert d["bonus"][0] == am[walk[-1]]


def _relaxed_case():
    import workload
    return workload.build(0, exercise=True, poison_tail=False)


def test_relaxed_reduces_to_strict_for_k1_tau0_phi0():
    case = _relaxed_case()
    w = case.w
    strict_w = synth.Workload(**{**w.__dict__})
    strict_w.src = np.zeros_like(w.src)
    strict = oracle.decide(strict_w, case.z)
    for p in (synth.AcceptParams(topk=1), synth.AcceptParams(max_relaxed=0)):
        d = oracle.decide(w, case.z, p)
        np.testing.assert_array_equal(d["acc_len"], strict["acc_len"])
        np.testing.assert_array_equal(d["path"], strict["path"])
    # tau = 0: only exact greedy tokens have a zero gap (the margins keep others >= 1e-3 away)
    d = oracle.decide(w, case.z, synth.AcceptParams(tau=0.0))
    np.testing.assert_array_equal(d["acc_len"], strict["acc_len"])


def test_config0_workload_exercises_relaxed_acceptance():
    case = _relaxed_case()
    d = case.expected
    assert ((d["flags"] & oracle.FLAG_RELAXED) & ~(d["flags"] & oracle.FLAG_GREEDY)).any()
    assert d["acc_len"][0] >= 1
