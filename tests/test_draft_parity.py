"""Parity of the library's drafting side (C++, include/respec_draft.h) with the
oracle (oracle/draft.py) on seeded inputs: trigger decisions and values,
retrieval positions from the suffix automaton, EMA selection and scores,
BuildDraftTree and whole sessions of Algorithm 1.  Integer outputs and
decisions are compared exactly; scores are double on both sides with the same
operation order and are compared exactly too.  These run on the host: the
drafting side never touches a GPU.
"""
import math
import os
import re

import numpy as np
import pytest

from oracle import draft as od
from paper_2511_01282_amd import binding, draft

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

pytestmark = pytest.mark.skipif(not os.path.exists(binding.LIB_PATH), reason="library not built")


def f32(x):
    return float(np.float32(x))


def test_library_exports_every_declared_drafting_call():
    text = open(os.path.join(ROOT, "include", "respec_draft.h")).read()
    declared = set(re.findall(r"\b(respec_\w+)\s*\(", text))
    assert declared == set(draft.DRAFT_EXPORTS)
    L = draft.lib()
    for name in declared:
        assert hasattr(L, name), name


def test_trigger_parity():
    rng = np.random.default_rng(10)
    for _ in range(3000):
        n = int(rng.integers(0, 9))
        ent = rng.choice([0.25, 0.5, 1.0, 1.5, 2.0], size=n) if rng.random() < 0.4 else rng.uniform(0, 4, n)
        ent = ent.astype(np.float32)
        if n and rng.random() < 0.15:
            ent[int(rng.integers(0, n))] = np.nan
        l = int(rng.integers(1, 7))
        lam = f32(rng.choice([0.0, 0.5, -0.25, rng.uniform(-1, 2)]))
        theta = f32(rng.choice([1.5, rng.uniform(0, 3)]))
        g = draft.trigger_eval(ent, l, lam, theta)
        k, h, c, fire = od.trigger_eval([float(x) for x in ent], l, lam, theta)
        assert (g.key_len, g.fire) == (k, fire)
        if k:
            assert g.h_min == f32(h) and g.c_min == f32(c)
        else:
            assert math.isnan(g.h_min) and math.isnan(g.c_min)


def test_trigger_errors():
    with pytest.raises(binding.VerifyError):
        draft.trigger_eval([1.0], max_lookback=0)
    with pytest.raises(binding.VerifyError):
        draft.trigger_eval([1.0], lambda_e=float("inf"))


def test_sam_positions_parity_incremental():
    rng = np.random.default_rng(11)
    for trial in range(40):
        alpha = int(rng.integers(1, 6))
        sam = draft.Sam()
        text = []
        for _ in range(int(rng.integers(1, 12))):
            chunk = [int(x) for x in rng.integers(0, alpha, int(rng.integers(0, 40)))]
            sam.extend(chunk)
            text += chunk
            assert len(sam) == len(text)
            assert sam.text().tolist() == text
            for _ in range(8):
                k = int(rng.integers(1, 6))
                if text and rng.random() < 0.5:
                    key = text[max(0, len(text) - k):]
                else:
                    key = [int(x) for x in rng.integers(0, alpha + 1, k)]
                assert sam.positions(key).tolist() == od.positions(text, key)
                cap = int(rng.integers(0, 4))
                assert sam.positions(key, cap).tolist() == od.positions(text, key)[:cap]


def test_sam_large_alphabet_and_long_context():
    rng = np.random.default_rng(12)
    base = [int(x) for x in rng.integers(0, 128256, 3000)]
    text = base + base[500:900] + [int(x) for x in rng.integers(0, 50, 2000)] + base[100:300]
    sam = draft.Sam(text)
    for start in range(0, len(text) - 4, 97):
        for k in (1, 2, 3):
            key = text[start:start + k]
            assert sam.positions(key).tolist() == od.positions(text, key)


def test_sam_errors():
    sam = draft.Sam([1, 2, 3])
    with pytest.raises(binding.VerifyError):
        sam.extend([4, -1])
    assert sam.text().tolist() == [1, 2, 3, 4]          # tokens before the bad one were appended
    with pytest.raises(binding.VerifyError):
        sam.positions([])
    with pytest.raises(binding.VerifyError):
        sam.text(2, 5)


def test_selection_and_ema_parity():
    rng = np.random.default_rng(13)
    for trial in range(30):
        alpha = f32(rng.choice([0.5, 0.25, rng.uniform(0, 1)]))
        theta, s0 = f32(rng.uniform(0, 0.5)), f32(rng.choice([0.5, rng.uniform(0, 1)]))
        n_select = int(rng.integers(1, 6))
        kw = dict(alpha=alpha, theta_score=theta, s0=s0, n_select=n_select)
        sc_lib, sc_or = draft.Scores(), {}
        for step in range(60):
            pos = sorted(set(int(x) for x in rng.integers(0, 40, int(rng.integers(0, 12)))), reverse=True)
            sel = sc_lib.select(pos, **kw).tolist()
            assert sel == od.select(sc_or, pos, alpha, theta, s0, n_select)
            if not sel:
                continue
            l_draft = [int(x) for x in rng.integers(1, 9, len(sel))]
            winner = int(rng.integers(-1, len(sel)))
            l_acc = int(rng.integers(0, l_draft[winner] + 1)) if winner >= 0 else 0
            sc_lib.update(sel, winner, l_acc, l_draft, **kw)
            od.ema_update(sc_or, sel, winner, l_acc, l_draft, alpha, s0)
            assert len(sc_lib) == len(sc_or)
            for p, v in sc_or.items():
                assert sc_lib.get(p, s0) == v


def test_negative_positions_are_rejected():
    sc = draft.Scores()
    with pytest.raises(binding.VerifyError):
        sc.select([3, -1])
    with pytest.raises(binding.VerifyError):
        sc.update([-2], -1, 0, None)
    assert len(sc) == 0


def test_ema_update_errors():
    sc = draft.Scores()
    with pytest.raises(binding.VerifyError):
        sc.update([1, 2], 2, 0, [1, 1])                # winner out of range
    with pytest.raises(binding.VerifyError):
        sc.update([1, 2], 0, 3, [2, 2])                # accepted more than drafted
    with pytest.raises(binding.VerifyError):
        sc.update([1], 0, 0, [1], alpha=1.5)
    assert len(sc) == 0


def test_build_tree_parity():
    rng = np.random.default_rng(14)
    for _ in range(300):
        n = int(rng.integers(1, 120))
        text = [int(x) for x in rng.integers(0, int(rng.integers(1, 5)), n)]
        sam = draft.Sam(text)
        sel = sorted(set(int(x) for x in rng.integers(0, n, int(rng.integers(0, 8)))), reverse=True)
        rng.shuffle(sel)
        dlen, max_nodes = int(rng.integers(1, 25)), int(rng.integers(2, 129))
        t = draft.build_tree(sam, sel, dlen, max_nodes)
        parent, token, src, ce, cl = od.build_tree(text, sel, dlen, max_nodes)
        assert t.parent.tolist() == parent and t.token.tolist() == token and t.src.tolist() == src
        assert t.cand_end.tolist() == ce and t.cand_len.tolist() == cl
        assert binding.check_tree(t.parent, 64) == binding.OK


def _run_sessions(seed, steps, **kw):
    """Drive the library and oracle sessions with the same random verification outcomes."""
    rng = np.random.default_rng(seed)
    lib_s, or_s = draft.DraftSession(**kw), od.Session(**kw)
    alpha = int(rng.integers(2, 6))
    prompt = [int(x) for x in rng.integers(0, alpha, int(rng.integers(1, 40)))]
    pe = rng.uniform(0, 2, len(prompt)).astype(np.float32)
    pe[0] = np.nan
    lib_s.append(prompt, pe)
    or_s.append(prompt, [float(x) for x in pe])
    n_retrieved = 0
    for _ in range(steps):
        p = lib_s.propose()
        r = or_s.propose()
        assert p.retrieved == r["retrieved"]
        assert (p.trigger.key_len, p.trigger.fire) == r["trigger"][0:1] + (r["trigger"][3],)
        assert p.n_positions == r["n_positions"]
        assert p.selected.tolist() == r["selected"]
        assert p.tree.parent.tolist() == r["parent"] and p.tree.token.tolist() == r["token"]
        assert p.tree.src.tolist() == r["src"]
        assert p.tree.cand_end.tolist() == r["cand_end"] and p.tree.cand_len.tolist() == r["cand_len"]
        n_retrieved += p.retrieved
        # a random verification outcome: a prefix of a random root-to-node chain
        parent, token = list(r["parent"]), list(r["token"])
        if not p.retrieved:   # stand-in for the model drafter: a random chain
            for _ in range(int(rng.integers(0, 4))):
                parent.append(len(parent) - 1)
                token.append(int(rng.integers(0, alpha)))
        v = int(rng.integers(0, len(parent)))
        chain = []
        while v >= 0:
            chain.append(v)
            v = parent[v]
        chain.reverse()
        acc = int(rng.integers(0, len(chain)))
        path = chain[:acc + 1] + [-1] * 3
        ent = rng.uniform(0, 2.5, len(parent)).astype(np.float32)
        bonus = int(rng.integers(0, alpha))
        lib_s.commit(np.array(token, np.int32), path, acc, bonus, ent)
        or_s.commit(token, path, acc, bonus, [float(x) for x in ent])
        assert lib_s.sam.text().tolist() == or_s.text
        assert len(lib_s.scores) == len(or_s.scores)
        for q, val in or_s.scores.items():
            assert lib_s.scores.get(q, kw.get("s0", 0.5)) == val
    return n_retrieved


@pytest.mark.parametrize("seed", range(6))
def test_session_parity(seed):
    kw = [dict(), dict(max_lookback=2, lambda_e=0.25, theta_entropy=2.0, alpha=0.25, theta_score=0.2, n_select=2,
                       max_draft_len=6, max_nodes=12),
          dict(max_lookback=4, lambda_e=0.0, theta_entropy=1.0, alpha=0.75, theta_score=0.3, s0=0.625,
               n_select=5, max_draft_len=3, max_nodes=128)][seed % 3]
    assert _run_sessions(100 + seed, 80, **kw) > 0


def test_session_commit_rejects_a_path_outside_the_proposal():
    s = draft.DraftSession(theta_entropy=10.0)
    s.append([1, 2, 3, 1, 2, 3, 1, 2], np.full(8, 0.5, np.float32))
    p = s.propose()
    assert p.retrieved and len(p.tree.parent) > 2
    bad = [0, 2]                                         # node 2's parent is node 1
    with pytest.raises(binding.VerifyError):
        s.commit(p.tree.token, bad, 1, 0, np.zeros(len(p.tree.parent), np.float32))
    s.commit(p.tree.token, [0, 1, 2], 2, 0, np.zeros(len(p.tree.parent), np.float32))
    assert s.sam.text().tolist() == [1, 2, 3, 1, 2, 3, 1, 2, 3, 1, 0]
