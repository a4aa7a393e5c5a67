"""The C ABI on the host: exports, plan creation, and argument validation.

None of these calls reaches the GPU: every step call here is rejected by the
host checks before a kernel is enqueued (fake device addresses are never
dereferenced on the host).
"""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "respec_verify.h")


@pytest.fixture(scope="module")
def b():
    from paper_2511_01282_amd import binding
    if not os.path.exists(binding.LIB_PATH):
        from paper_2511_01282_amd import build
        build.build()
    binding.lib()
    return binding


def _header_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(respec_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_function(b):
    declared = _header_functions()
    assert set(declared) == set(b.EXPORTS)
    for name in declared:
        assert hasattr(b.lib(), name), name


def test_library_exports_the_measurement_probes(b):
    text = open(os.path.join(ROOT, "include", "respec_probe.h")).read()
    names = sorted(set(re.findall(r"\b(respec_probe_[a-z_]+)\s*\(", text)))
    assert names == ["respec_probe_mfma", "respec_probe_read"]
    for name in names:
        assert hasattr(b.lib(), name), name


def test_probes_reject_bad_arguments_before_launch(b):
    L = b.lib()
    L.respec_probe_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int32, ctypes.c_int32,
                                    ctypes.c_void_p, ctypes.c_void_p]
    L.respec_probe_mfma.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                    ctypes.c_void_p]
    assert L.respec_probe_read(FAKE, 4096 * 8, 8, 3, FAKE, None) == 1          # depth
    assert L.respec_probe_read(FAKE, 4096 * 8 + 16, 8, 8, FAKE, None) == 1     # not whole steps
    assert L.respec_probe_read(FAKE + 8, 4096 * 8, 8, 8, FAKE, None) == 1      # alignment
    assert L.respec_probe_read(None, 4096 * 8, 8, 8, FAKE, None) == 1
    assert L.respec_probe_mfma(0, 10, 0, FAKE, None) == 1
    assert L.respec_probe_mfma(8, 10, 2, FAKE, None) == 1
    assert L.respec_probe_mfma(8, 10, 0, None, None) == 1


def test_status_strings(b):
    for code in range(11):
        assert b.status_string(code)
    assert b.status_string(0) == "ok"


@pytest.mark.parametrize("parent,depth,code", [
    ([-1], 0, 0), ([-1, 0, 1, 1, 0], 2, 0), ([0], 3, 5), ([-1, 1], 3, 5), ([-1, 0, 3, 1], 3, 5),
    ([-1, 0, 1, 2], 2, 5), ([], 3, 2), (list(range(-1, 128)), 200, 2),
])
def test_check_tree(b, parent, depth, code):
    assert b.check_tree(parent, depth) == code


def _shape(b, **over):
    d = dict(hidden=4096, n_q_heads=32, n_kv_heads=32, head_dim=128, vocab=32000, dtype=b.BF16,
             max_batch=1, max_nodes=26, max_depth=6, max_kv_len=2048, topk_out=8)
    d.update(over)
    return b.Shape(*[d[f] for f, _ in b.Shape._fields_])


def _create(b, shape):
    h = ctypes.c_void_p()
    st = b.lib().respec_verify_create(ctypes.byref(shape), ctypes.byref(h))
    return st, h


@pytest.mark.parametrize("over,code", [
    ({}, 0), (dict(dtype=7), 3), (dict(head_dim=96, hidden=32 * 96), 2), (dict(n_kv_heads=5), 2),
    (dict(hidden=4000), 2), (dict(topk_out=0), 2), (dict(topk_out=17), 2), (dict(vocab=4), 2),
    (dict(max_nodes=129), 2), (dict(max_nodes=0), 2), (dict(max_depth=65), 2), (dict(max_batch=0), 2),
    (dict(max_kv_len=-1), 2), (dict(dtype=0, hidden=64, n_q_heads=1, n_kv_heads=1, head_dim=64), 2),
])
def test_create_validates_shape(b, over, code):
    st, h = _create(b, _shape(b, **over))
    assert st == code
    if st == 0:
        assert b.lib().respec_verify_workspace_bytes(h) > 0
        b.lib().respec_verify_destroy(h)
    else:
        assert not h.value


def test_workspace_grows_with_capacity(b):
    _, h1 = _create(b, _shape(b))
    _, h2 = _create(b, _shape(b, max_batch=8, max_nodes=32, max_kv_len=8192))
    L = b.lib()
    assert L.respec_verify_workspace_bytes(h2) > L.respec_verify_workspace_bytes(h1)
    assert L.respec_verify_workspace_bytes(None) == 0
    L.respec_verify_destroy(h1)
    L.respec_verify_destroy(h2)
    L.respec_verify_destroy(None)


FAKE = 0x7F0000000000  # 256-byte aligned fake device address; never dereferenced on the host


def _args(b, **over):
    a = b.Args()
    a.batch, a.total_nodes, a.max_nodes_in_batch, a.max_kv_len_in_batch = 1, 26, 26, 2048
    a.kv_capacity, a.stop_after = 2074, 0
    a.accept = b.AcceptParams(8, 3.0, 2, 2, 0, 1.0)
    for f in b.INPUT_FIELDS + b.OUTPUT_FIELDS:
        setattr(a, f, FAKE)
    for k, v in over.items():
        if k in ("topk", "tau", "min_lookahead", "max_relaxed", "stochastic", "temperature"):
            setattr(a.accept, k, v)
        else:
            setattr(a, k, v)
    return a


@pytest.mark.parametrize("over,code", [
    (dict(stop_after=4), 4), (dict(stop_after=-1), 4), (dict(batch=-1), 2), (dict(batch=2), 6),
    (dict(topk=0), 4), (dict(topk=9), 4), (dict(tau=-1.0), 4), (dict(tau=float("nan")), 4),
    (dict(tau=float("inf")), 4), (dict(min_lookahead=-1), 4), (dict(max_relaxed=-1), 4),
    (dict(max_nodes_in_batch=0), 2), (dict(max_nodes_in_batch=27), 6), (dict(max_kv_len_in_batch=4096), 6),
    (dict(total_nodes=0), 2), (dict(total_nodes=27), 2), (dict(kv_capacity=2073), 2),
    (dict(hidden=None), 1), (dict(k_cache=None), 1), (dict(parent=None), 1), (dict(lm_head=None), 1),
    (dict(logits=None), 1), (dict(token=None), 1), (dict(flags=None), 1), (dict(seq_status=None), 1),
    (dict(hidden=FAKE + 8), 2), (dict(lm_head=FAKE + 4), 2), (dict(logits=FAKE + 4), 2),
    # stochastic verification: mode, temperature, uniforms, draft distribution alignment
    (dict(stochastic=2), 4), (dict(stochastic=1, temperature=0.0), 4), (dict(stochastic=1, temperature=-1.0), 4),
    (dict(stochastic=1, temperature=float("inf")), 4), (dict(stochastic=1, temperature=float("nan")), 4),
    (dict(stochastic=1, uniform=None), 1), (dict(stochastic=1, draft_prob=FAKE + 4), 2),
])
def test_step_rejects_bad_arguments_before_launch(b, over, code):
    _, h = _create(b, _shape(b))
    a = _args(b, **over)
    assert b.lib().respec_verify_step(h, ctypes.byref(a), FAKE, None) == code
    b.lib().respec_verify_destroy(h)


def test_step_rejects_bad_workspace_and_null_plan(b):
    _, h = _create(b, _shape(b))
    a = _args(b)
    L = b.lib()
    assert L.respec_verify_step(h, ctypes.byref(a), None, None) == 8
    assert L.respec_verify_step(h, ctypes.byref(a), FAKE + 16, None) == 8
    assert L.respec_verify_step(None, ctypes.byref(a), FAKE, None) == 1
    assert L.respec_verify_step(h, None, FAKE, None) == 1
    assert L.respec_verify_workspace_init(h, FAKE + 8, None) == 8
    assert L.respec_verify_workspace_init(None, FAKE, None) == 1
    L.respec_verify_destroy(h)


def test_attention_only_step_needs_no_logit_buffers(b):
    # stop_after = ATTN with no LM head / logits pointers passes the NULL checks;
    # an out-of-range accept parameter is then ignored, so only a later check fails
    _, h = _create(b, _shape(b))
    a = _args(b, stop_after=1, lm_head=None, logits=None, topk=0, kv_capacity=10)
    assert b.lib().respec_verify_step(h, ctypes.byref(a), FAKE, None) == 2
    b.lib().respec_verify_destroy(h)


def test_statistics_only_step_needs_no_path_buffers(b):
    # stop_after = STATS: the path outputs may be NULL (the alignment check after the
    # NULL checks then fails, so nothing is launched), but the statistics and flags may not
    _, h = _create(b, _shape(b))
    none = dict(leaf_acc_len=None, path=None, acc_len=None, bonus=None, winner_leaf=None, seq_status=None,
                sample=None, hidden=FAKE + 8)
    a = _args(b, stop_after=3, **none)
    assert b.lib().respec_verify_step(h, ctypes.byref(a), FAKE, None) == 2
    for f in ("flags", "entropy", "topk_id", "token"):
        a = _args(b, stop_after=3, **dict(none, **{f: None}))
        assert b.lib().respec_verify_step(h, ctypes.byref(a), FAKE, None) == 1, f
    # the statistics level still checks the acceptance parameters (the predicates use them)
    a = _args(b, stop_after=3, topk=0)
    assert b.lib().respec_verify_step(h, ctypes.byref(a), FAKE, None) == 4
    b.lib().respec_verify_destroy(h)


def test_noalloc_step_checks_before_any_device_call(b):
    L = b.lib()
    a = _args(b)
    assert L.respec_verify_step_noalloc(None, ctypes.byref(a), None) == 1
    _, h = _create(b, _shape(b))
    assert L.respec_verify_step_noalloc(h, None, None) == 1
    L.respec_verify_destroy(h)
    # a plan whose workspace exceeds the static scratch is refused on the host
    _, big = _create(b, _shape(b, max_batch=64, max_nodes=128, max_kv_len=32768, vocab=128256, n_kv_heads=8))
    assert L.respec_verify_workspace_bytes(big) > b.NOALLOC_SCRATCH_BYTES
    assert L.respec_verify_step_noalloc(big, ctypes.byref(a), None) == b.ERR_SCRATCH
    L.respec_verify_destroy(big)
    st, many = _create(b, _shape(b, max_batch=b.NOALLOC_MAX_BATCH + 1, max_nodes=1, max_kv_len=16, vocab=64,
                                 hidden=256, n_q_heads=2, n_kv_heads=2))
    assert st == 0
    assert L.respec_verify_step_noalloc(many, ctypes.byref(a), None) == b.ERR_SCRATCH
    L.respec_verify_destroy(many)


def test_empty_batch_is_a_no_op(b):
    _, h = _create(b, _shape(b))
    a = _args(b, batch=0, total_nodes=0)
    assert b.lib().respec_verify_step(h, ctypes.byref(a), FAKE, None) == 0
    b.lib().respec_verify_destroy(h)
