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
    from paper_2511_01282_amd import runner
    plan = runner.make_plan(dl.workload(m, [0, 0], [-1], [0], [0]), "cuda:0", max_nodes=m.shape.max_nodes,
                            max_kv_len=4096)

    def verify(w):
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
