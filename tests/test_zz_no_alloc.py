"""The allocation-free entry point against the ordinary one, through the C ABI.

respec_verify_step_noalloc runs the same kernels as respec_verify_step with the
library's static scratch in place of the caller's workspace, so every output
must be identical bit for bit.  Two calls in a row, the second on a smaller
workload (fewer nodes, shorter cache, another plan, so another workspace
layout over the same scratch), check that one call's leftovers in the shared
array do not leak into the next.  A plan whose workspace exceeds the scratch
is refused on the host.
"""
import numpy as np
import pytest

import respec_synth as synth
import workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def rt():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2511_01282_amd import binding, runner
    binding.lib()
    return runner


def _run(rt, case, noalloc):
    import torch
    from paper_2511_01282_amd import binding
    w = case.w
    kw = rt.step_kwargs(w)
    plan = rt.make_plan(w, "cuda:0", max_kv_len=kw["max_kv_len_in_batch"])
    inputs = rt.upload(w, "cuda:0")
    s = w.shape
    out = binding.alloc_outputs(total_nodes=kw["total_nodes"], batch=kw["batch"], hidden=s.hidden,
                                vocab=s.vocab, topk_out=s.topk_out, max_depth=s.max_depth, device="cuda:0")
    for v in out.values():
        if v is not None:
            v.fill_(-7 if v.dtype != torch.uint8 else 0xEE)
    plan.step(inputs, out, noalloc=noalloc, **kw)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items() if v is not None}


def _same(a, b, label):
    for k in a:
        np.testing.assert_array_equal(a[k], b[k], err_msg=f"{label}: {k}")


@pytest.mark.timeout(600)
def test_noalloc_matches_the_workspace_entry_point_twice(rt):
    big = workload.build(1)              # 26-node tree, KV length 2048, 7B shapes
    small = workload.build(0)            # 16-node tree, KV length 512, float32 (another layout)
    for label, case in (("first call, 26 nodes", big), ("second call, 16 nodes", small)):
        print(f"[noalloc] {label}", flush=True)
        ref = _run(rt, case, noalloc=False)
        got = _run(rt, case, noalloc=True)
        _same(got, ref, label)
        e = case.expected
        for k in ("argmax", "flags", "path", "acc_len", "bonus", "winner_leaf", "seq_status"):
            np.testing.assert_array_equal(got[k], e[k], err_msg=f"{label}: {k} against the oracle")


@pytest.mark.timeout(600)
def test_noalloc_smaller_batch_after_larger(rt):
    # a ragged 4-sequence batch, then a 2-sequence batch with fewer nodes: the
    # completion counters of sequences 2 and 3 must be back at zero
    shp = synth.Shape("edge", "bf16", 8 * 128, 8, 2, 128, 3000, 4, 13, 12, 8)
    parents = [[-1, 0, 1, 1, 3], [-1], [-1] + list(range(0, 12)), [-1, 0, 0, 0]]
    w = synth.custom(shp, parents, [33, 1, 200, 97], seed=303, poison_tail=True)
    first = workload.finish(w)
    shp2 = synth.Shape("edge", "bf16", 8 * 128, 8, 2, 128, 3000, 2, 4, 12, 8)
    # (the longest prefix goes with the largest tree: the cache holds max prefix + max nodes rows)
    w2 = synth.custom(shp2, [[-1, 0, 0, 2], [-1, 0, 1]], [20, 5], seed=304, poison_tail=True)
    second = workload.finish(w2)
    for label, case in (("4 sequences", first), ("2 sequences", second)):
        print(f"[noalloc] {label}", flush=True)
        ref = _run(rt, case, noalloc=False)
        got = _run(rt, case, noalloc=True)
        _same(got, ref, label)
        np.testing.assert_array_equal(got["acc_len"], case.expected["acc_len"], err_msg=label)


@pytest.mark.timeout(600)
def test_noalloc_gemm_lm_head_and_shared_tile_attention(rt):
    # 218 token rows in two trees (the LM head's GEMM form), then a grouped-query
    # batch on the shared-tile attention (8 query heads per KV head), then the
    # first again: three plans in a row over one scratch
    shp = synth.Shape("edge", "bf16", 4 * 64, 4, 2, 64, 3001, 2, 128, 8, 8)
    parents = [[-1] + [(j - 1) // 3 for j in range(1, 128)], [-1] + [(j - 1) // 2 for j in range(1, 90)]]
    gemm = workload.finish(synth.custom(shp, parents, [300, 90], seed=505, poison_tail=True))
    shp2 = synth.Shape("edge", "bf16", 16 * 128, 16, 2, 128, 4000, 2, 40, 12, 8)
    parents2 = [[-1] + [max(0, j - 4) for j in range(1, 40)], [-1, 0, 1, 1]]
    gqa = workload.finish(synth.custom(shp2, parents2, [700, 60], seed=506, poison_tail=True))
    for label, case in (("218 rows", gemm), ("grouped-query", gqa), ("218 rows again", gemm)):
        print(f"[noalloc] {label}", flush=True)
        ref = _run(rt, case, noalloc=False)
        got = _run(rt, case, noalloc=True)
        _same(got, ref, label)
        e = case.expected
        for k in ("argmax", "flags", "path", "acc_len", "bonus", "winner_leaf", "seq_status"):
            np.testing.assert_array_equal(got[k], e[k], err_msg=f"{label}: {k} against the oracle")


def test_noalloc_refuses_a_plan_beyond_the_scratch(rt):
    import torch
    from paper_2511_01282_amd import binding
    # a plan for 64 sequences of 128 nodes at KV length 32768 needs far more than 64 MiB
    plan = binding.Plan(hidden=4096, n_q_heads=32, n_kv_heads=8, head_dim=128, vocab=128256, dtype=binding.BF16,
                        max_batch=64, max_nodes=128, max_depth=8, max_kv_len=32768, topk_out=8, device="cuda:0")
    assert plan.workspace_bytes > binding.NOALLOC_SCRATCH_BYTES
    z = torch.zeros(16, dtype=torch.int32, device="cuda:0")
    with pytest.raises(binding.VerifyError) as ei:
        plan.step({"node_off": z, "kv_len": z, "hidden": z, "k_cache": z, "v_cache": z, "lm_head": z,
                   "parent": z, "token": z, "src": z}, {}, batch=1, total_nodes=1, max_nodes_in_batch=1,
                  max_kv_len_in_batch=0, kv_capacity=1, noalloc=True)
    assert ei.value.status == binding.ERR_SCRATCH
