"""GPU parity of stochastic (lossless speculative-sampling) verification.

The HIP path with accept.stochastic = 1 against the oracle's stochastic
verification, on the same logits, drafter distributions and uniforms.  The
uniforms keep every decision away from its threshold (tests/workload.py), so
the accept bits, residual draws, walked paths, bonus tokens and per-leaf
lengths must agree exactly; the statistics are those of the ordinary step.
"""
import numpy as np
import pytest

import respec_synth as synth
import workload

from test_gpu_parity import compare, _edge_shape

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def rt():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2511_01282_amd import binding, runner
    binding.lib()
    return runner


CASES = {
    # name: (config or custom tree spec, temperature, drafter distributions given)
    "c0-T1": (0, 1.0, True),
    "c1-T0.7": (1, 0.7, True),
    "c1-deterministic-T1.3": (1, 1.3, False),
    "c2-T1": (2, 1.0, True),
    "c3-T1": (3, 1.0, True),
    "c4-T1": (4, 1.0, True),
    "star30-T1.5": ("star", 1.5, True),
    "ragged-T0.9": ("ragged", 0.9, True),
    "odd-vocab-T1.1": ("odd", 1.1, True),
    "drafter-equals-target-T0.3": ("exact", 0.3, True),
}


def _custom(kind):
    if kind in ("odd", "exact"):
        v = 3001 if kind == "odd" else 3000
        shp = synth.Shape("edge", "bf16", 4 * 64, 4, 1, 64, v, 2, 8, 8, 8)
        parents = [[-1, 0, 1, 1, 3, 0, 5, 5], [-1, 0, 0, 2]]
        w = synth.custom(shp, parents, [70, 40], seed=211, poison_tail=True,
                         src=[[0] + [j % 2 for j in range(1, len(p))] for p in parents])
        return workload.finish(w)
    if kind == "star":
        shp = _edge_shape("bf16", 4, 2, 128)
        parents, kv = [[-1] + [0] * 30], [130]
    else:
        shp = _edge_shape("bf16", 8, 2, 128)
        parents = [[-1, 0, 1, 1, 3], [-1], [-1] + list(range(0, 12)), [-1, 0, 0, 0]]
        kv = [33, 1, 200, 97]
    w = synth.custom(shp, parents, kv, seed=303, poison_tail=True,
                     src=[[0] + [j % 2 for j in range(1, len(p))] for p in parents])
    w.shape = synth.Shape("edge", "bf16", shp.hidden, shp.n_q_heads, shp.n_kv_heads, shp.head_dim, shp.vocab,
                          len(parents), max(len(p) for p in parents), 12, 8)
    return workload.finish(w)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", list(CASES))
def test_stochastic_parity(rt, name):
    import torch
    spec, T, with_q = CASES[name]
    print(f"[stochastic {name}] building case", flush=True)
    case = workload.build(spec) if isinstance(spec, int) else _custom(spec)
    # "exact": the drafter's distributions are the target's own (every model draft passes)
    q, u = workload.stochastic_inputs(case, T, with_q=with_q, q_noise=0.0 if spec == "exact" else 0.5)
    exp = workload.stochastic_expected(case, q, u, T)
    case.expected = dict(case.expected, **exp)
    case.w.params = synth.AcceptParams(case.w.params.topk, case.w.params.tau, case.w.params.min_lookahead,
                                       case.w.params.max_relaxed, 1, T)
    inputs = rt.upload(case.w, "cuda:0")
    inputs["draft_prob"] = torch.from_numpy(q).to("cuda:0") if q is not None else None
    inputs["uniform"] = torch.from_numpy(u).to("cuda:0")
    print(f"[stochastic {name}] running GPU step: acc_len={exp['acc_len'].tolist()}", flush=True)
    out = rt.run(case.w, inputs=inputs, device="cuda:0")
    compare(case, out, f"stochastic {name}")
    np.testing.assert_array_equal(out["sample"], exp["sample"], err_msg="sample")
    # the walk accepted something somewhere, and drew somewhere
    assert (exp["sample"] >= 0).any()
