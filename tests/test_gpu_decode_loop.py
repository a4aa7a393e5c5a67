"""Algorithm 1's decoding loop on the GPU path against the oracle.

The library's drafting session (trigger, suffix-automaton retrieval, EMA
selection, BuildDraftTree, feedback) and the HIP verification step run the
loop; the oracle's session and verification step run it beside them on the
same token-conditioned proxy target.  Each step's proposal, accepted path and
the generated text must agree exactly.  Under strict verification the loop
must also reproduce plain greedy decoding.
"""
import numpy as np
import pytest

import oracle
import respec_synth as synth
from oracle import draft as od

import decode_loop as dl

pytestmark = pytest.mark.gpu


class _LibSession:
    def __init__(self, **kw):
        from paper_2511_01282_amd import draft
        self.s = draft.DraftSession(**kw)

    def append(self, t, e):
        self.s.append(t, e)

    def propose(self):
        p = self.s.propose()
        return p.tree.parent, p.tree.token, p.tree.src, p.retrieved

    def commit(self, token, path, acc, bonus, ent):
        self.s.commit(token, path, acc, bonus, ent)

    def text(self):
        return self.s.sam.text().tolist()


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


def _gpu_verify(m):
    # Every step's decisions (argmax gaps, tau and rank-k boundaries) must sit at
    # least MARGIN away from their thresholds in the oracle's logits of that step,
    # so float32 differences between the two paths cannot flip one: a near-tie is
    # reported as such instead of surfacing as a divergence of the loops.
    import workload
    from paper_2511_01282_amd import runner
    plan = runner.make_plan(dl.workload(m, [0, 0], [-1], [0], [0]), "cuda:0", max_nodes=m.shape.max_nodes,
                            max_kv_len=4096)
    count = [0]

    def verify(w):
        margin = workload.min_decision_margin(w, oracle.forward(w)["z"])
        assert margin >= workload.MARGIN, f"step {count[0]}: a decision is {margin:.2e} from its threshold"
        count[0] += 1
        return runner.run(w, plan=plan, device="cuda:0", attn_out=False)
    return verify


@pytest.mark.parametrize("params", [synth.AcceptParams(topk=1, tau=0.0), synth.AcceptParams(topk=8, tau=3.0)],
                         ids=["strict", "relaxed"])
def test_decode_loop_matches_the_oracle(params):
    m = dl.make_model(params=params)
    pr = dl.prompt()
    print(f"[loop] {params}", flush=True)
    g_text, g_steps = dl.speculative_decode(m, _LibSession(), pr, 60, _gpu_verify(m))
    o_text, o_steps = dl.speculative_decode(m, _OracleSession(), pr, 60, oracle.verify_step)
    assert g_steps == o_steps
    assert g_text == o_text
    assert sum(r for r, _, _ in g_steps) >= 3
    if params.topk == 1:
        assert g_text == dl.greedy_decode(m, pr, len(g_text) - len(pr), oracle.verify_step)


def test_stochastic_decode_loop_in_lockstep():
    # Algorithm 1 with speculative-sampling verification (temperature 0.5):
    # at every step both sessions propose the same tree, the uniforms are
    # drawn with decision margins from the oracle's logits of that step, and
    # the GPU's sampled walk, bonus token and per-node draws must equal the
    # oracle's.  Both sessions then commit the same outcome.
    import torch
    import workload
    from paper_2511_01282_amd import runner

    T = 0.5
    m = dl.make_model(params=synth.AcceptParams(topk=8, tau=3.0, stochastic=1, temperature=T))
    pr = dl.prompt()
    lib, orc = _LibSession(), _OracleSession()
    lib.append(pr, None)
    orc.append(pr, None)
    plan = runner.make_plan(dl.workload(m, [0, 0], [-1], [0], [0]), "cuda:0", max_nodes=m.shape.max_nodes,
                            max_kv_len=4096)
    retrieved_steps, accepted = 0, 0
    for step in range(60):
        pl, po = lib.propose(), orc.propose()
        assert [list(x) for x in pl[:3]] == [list(x) for x in po[:3]] and pl[3] == po[3], step
        parent, token, src, retrieved = po
        w = dl.workload(m, orc.text(), parent, token, src)
        f = oracle.forward(w)
        case = workload.Case(w, f["z"], f["attn"], f["x"], oracle.decide(w, f["z"]))
        _, u = workload.stochastic_inputs(case, T, seed=1000 + step, with_q=False)
        exp = workload.stochastic_expected(case, None, u, T)
        inputs = runner.upload(w, "cuda:0")
        inputs["uniform"] = torch.from_numpy(u).to("cuda:0")
        out = runner.run(w, plan=plan, inputs=inputs, device="cuda:0", attn_out=False)
        for k in ("acc_len", "bonus", "path", "sample", "winner_leaf", "leaf_acc_len"):
            np.testing.assert_array_equal(out[k], exp[k], err_msg=f"step {step}: {k}")
        walk_bits = 16 | 32
        np.testing.assert_array_equal(out["flags"] & walk_bits, exp["flags"] & walk_bits, err_msg=f"step {step}")
        acc = int(exp["acc_len"][0])
        ent = case.expected["entropy"].astype(np.float32)
        lib.commit(np.asarray(token, np.int32), exp["path"][0], acc, int(exp["bonus"][0]), ent)
        orc.commit(token, exp["path"][0], acc, int(exp["bonus"][0]), ent)
        retrieved_steps += bool(retrieved)
        accepted += acc
    assert lib.text() == orc.text()
    assert retrieved_steps >= 5 and accepted >= 20
