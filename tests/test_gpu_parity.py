"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Same seeded inputs on both sides.  Bar:
  - integer and index outputs (argmax, flags, leaf/accepted lengths, paths,
    bonus, winner, status) bit-exact; top-k ids exact except where the
    oracle's float32 logits of the two ids are within 1e-4 (then both orders
    are valid and the id sets must still be valid top-k members);
  - float outputs (attention O, logits, max logit, lse, entropy, log-probs)
    within rtol 2e-2 / atol 1e-3 (bf16 inputs, fp32 accumulation); float32
    workloads additionally within 1e-4.
Every workload keeps acceptance decisions >= 1e-3 away from their thresholds
(see tests/workload.py), so the float differences cannot flip a decision.

The residual x = round(h + O) that feeds the LM head is compared bit for bit
(bf16) against the oracle's, which rounds the exact sum once: where they
differ, the GPU's value must still be the rounding of a sum within X_EPS of
the oracle's exact sum (the kernel's O differs from the oracle's by far less
than X_EPS), i.e. lie between round(pre - X_EPS) and round(pre + X_EPS).
That happens only next to a rounding midpoint, or for sums so close to zero
that bf16's spacing there is below X_EPS.
tok_rank is compared exactly wherever the oracle's logits are unambiguous
(no other logit within RANK_EPS, the logit tolerance, of the token's); where
one is, the GPU's rank must lie in the range those logits allow.  It must
also be exactly the rank of the token in the logits the GPU returned.
"""
import numpy as np
import pytest

import respec_synth as synth
import workload

pytestmark = pytest.mark.gpu

RTOL, ATOL = 2e-2, 1e-3
X_EPS = 1e-5      # bound on |O_gpu - O_oracle| (measured: < 1e-6) within which x may round either way
RANK_EPS = ATOL   # logits this close to the token's may order either way


@pytest.fixture(scope="module")
def rt():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2511_01282_amd import binding, runner
    binding.lib()
    return runner


def _say(msg):
    print(msg, flush=True)


def compare(case, out, label, check_float=True):
    # rows of sequences reported as malformed carry no defined values (the oracle gives
    # their nodes a stand-in ancestor set): only the integer outputs are compared there
    e = case.expected
    w = case.w
    z32 = case.z.astype(np.float32)
    valid = e["seq_status"][_seq_of(w)] == 0
    if check_float:
        if out.get("attn_out") is not None:
            err = np.abs(out["attn_out"][valid] - case.attn[valid]).max()
            _say(f"[{label}] max|dO| = {err:.3e}")
            np.testing.assert_allclose(out["attn_out"][valid], case.attn[valid], rtol=RTOL, atol=ATOL)
        err = np.abs(out["logits"][valid] - case.z[valid]).max()
        _say(f"[{label}] max|dz| = {err:.3e}")
        np.testing.assert_allclose(out["logits"][valid], case.z[valid], rtol=RTOL, atol=ATOL)
        for k in ("max_logit", "lse", "entropy"):
            np.testing.assert_allclose(out[k][valid], e[k][valid], rtol=RTOL, atol=ATOL, err_msg=k)
        np.testing.assert_allclose(out["topk_logprob"][valid], e["topk_logprob"][valid], rtol=RTOL, atol=ATOL)
        nonroot = np.array([w.parent[j] >= 0 for j in range(len(w.parent))]) & valid
        np.testing.assert_allclose(out["tok_logprob"][nonroot], e["tok_logprob"][nonroot], rtol=RTOL, atol=ATOL)
        if w.shape.dtype == "f32":
            np.testing.assert_allclose(out["logits"][valid], case.z[valid], rtol=1e-4, atol=1e-4)
            np.testing.assert_allclose(out["entropy"][valid], e["entropy"][valid], rtol=1e-4, atol=1e-4)
    np.testing.assert_array_equal(out["argmax"][valid], e["argmax"][valid], err_msg="argmax")
    gid, oid = out["topk_id"], e["topk_id"]
    for r, k in zip(*np.nonzero((gid != oid) & valid[:, None])):
        assert abs(float(z32[r, gid[r, k]]) - float(z32[r, oid[r, k]])) < 1e-4, (r, k)
    for name in ("flags", "leaf_acc_len", "path", "acc_len", "bonus", "winner_leaf", "seq_status"):
        np.testing.assert_array_equal(out[name], e[name], err_msg=name)
    if out.get("x_out") is not None:
        check_x(case, out["x_out"], label, valid)
    if out.get("tok_rank") is not None:
        check_rank(case, out["tok_rank"], out["logits"], label)


def check_x(case, x_out, label, valid=None):
    """x against the oracle's residual: bit-exact for bf16 up to near-midpoint sums."""
    w = case.w
    if valid is None:
        valid = np.ones(x_out.shape[0], bool)
    if w.shape.dtype != "bf16":
        np.testing.assert_allclose(x_out[valid].astype(np.float64), case.x[valid], rtol=1e-4, atol=1e-4,
                                   err_msg="x")
        return
    gpu = synth.bf16_bits_to_f32(x_out).astype(np.float64)
    diff = (gpu != case.x) & valid[:, None]
    n = int(diff.sum())
    if n:
        pre = (synth.bf16_bits_to_f32(w.hidden).astype(np.float64) + case.attn)[diff]
        lo, hi = _rne_bf16(pre - X_EPS), _rne_bf16(pre + X_EPS)
        g = gpu[diff]
        bad = (g < lo) | (g > hi)
        assert not bad.any(), (f"x differs at {int(bad.sum())} elements by more than a rounding of a sum "
                               f"within {X_EPS} of the exact one: gpu {g[bad][:4]}, oracle {case.x[diff][bad][:4]}, "
                               f"exact sum {pre[bad][:4]}")
    _say(f"[{label}] x bit-exact at {int(valid.sum()) * x_out.shape[1] - n} of {int(valid.sum()) * x_out.shape[1]} "
         f"elements ({n} sums within {X_EPS} of a rounding boundary)")


def _rne_bf16(d):
    """Nearest bf16 value (ties to even) of doubles d: d = m 2^e, spacing 2^(e-8)."""
    m, e = np.frexp(d)
    q = np.ldexp(1.0, np.maximum(e - 8, -133))
    return np.where(d == 0, 0.0, np.rint(d / q) * q)


def check_rank(case, rank, logits, label):
    """tok_rank: exact where the oracle's logits order the token unambiguously, else in range."""
    w, e = case.w, case.expected
    seq = _seq_of(w)
    z = case.z
    n_exact = n_range = 0
    for j in range(len(w.parent)):
        b = seq[j]
        if e["seq_status"][b] != 0 or w.parent[j] < 0:
            continue
        i = int(w.node_off[b]) + int(w.parent[j])
        t = int(w.token[j])
        zi, zt = z[i], z[i, t]
        lo = int((zi > zt + RANK_EPS).sum())
        hi = int((zi >= zt - RANK_EPS).sum()) - 1
        assert lo <= int(e["tok_rank"][j]) <= hi
        if lo == hi:
            assert rank[j] == e["tok_rank"][j], (label, j, rank[j], e["tok_rank"][j])
            n_exact += 1
        else:
            assert lo <= rank[j] <= hi, (label, j, rank[j], lo, hi)
            n_range += 1
        # the rank of the token in the logits the GPU returned
        g = logits[i]
        gt = g[t]
        assert rank[j] == int((g > gt).sum()) + int(((g == gt) & (np.arange(g.shape[0]) < t)).sum())
    roots = w.parent < 0
    assert (rank[roots] == -1).all()
    _say(f"[{label}] tok_rank exact at {n_exact} nodes, within the logit tolerance at {n_range}")


def _seq_of(w):
    seq = np.zeros(len(w.parent), np.int64)
    for b in range(len(w.node_off) - 1):
        seq[w.node_off[b]:w.node_off[b + 1]] = b
    return seq


# ---------------------------------------------------------------------------
# the five workload shapes, at full size
# ---------------------------------------------------------------------------

@pytest.mark.timeout(900)
@pytest.mark.parametrize("cfg", [0, 1, 2, 3, 4])
def test_config_parity(rt, cfg):
    _say(f"[config {cfg}] building case (seed {synth.SEED_BASE + cfg})")
    case = workload.build(cfg)
    _say(f"[config {cfg}] running GPU step: acc_len={case.expected['acc_len'].tolist()}")
    out = rt.run(case.w, x_out=True, tok_rank=True)
    compare(case, out, f"config {cfg}")


# ---------------------------------------------------------------------------
# edge cases
# ---------------------------------------------------------------------------

def _edge_shape(dtype, hq=4, hkv=2, d=128, v=3000, depth=8, topk_out=8):
    return synth.Shape("edge", dtype, hq * d, hq, hkv, d, v, 1, 128, depth, topk_out)


EDGE = {
    # name: (dtype, hq, hkv, d, parents, kv_len)
    "root-only+empty-prefix": ("bf16", 4, 2, 128, [[-1], [-1, 0]], [0, 0]),
    "ragged-batch": ("bf16", 8, 2, 128, [[-1, 0, 1, 1, 3], [-1], [-1] + list(range(0, 12)), [-1, 0, 0, 0]],
                     [33, 1, 200, 97]),
    "chain-causal-f32": ("f32", 2, 1, 64, [[-1] + list(range(0, 20))], [45]),
    "gqa8-star": ("bf16", 8, 1, 128, [[-1] + [0] * 30], [130]),
    "d64-bf16-mixed": ("bf16", 4, 4, 64, [[-1, 0, 1, 2, 0, 4, 5, 1, 7]], [64]),
    # 96 query rows per KV head (three waves sharing each KV tile), head_dim 64
    "d64-bf16-shared-rows": ("bf16", 4, 2, 64, [[-1] + [j // 2 for j in range(0, 47)]], [300]),
    # 136 query rows per KV head: one key group of five row waves, the last with one live
    # row block of two (head_dim 64 and 128; the split ends fall inside KV tiles)
    "d64-bf16-136-rows": ("bf16", 16, 2, 64, [[-1] + [max(0, j - 3) for j in range(1, 17)]], [500]),
    "d128-bf16-136-rows": ("bf16", 8, 1, 128, [[-1] + [j // 2 for j in range(0, 16)]], [777]),
    "max-nodes-128": ("bf16", 2, 2, 128, [[-1] + [max(0, j - 4) for j in range(1, 128)]], [31]),
    "max-depth-64": ("bf16", 2, 2, 128, [[-1] + list(range(0, 64))], [5]),
    # LM-head tiles of 48 and 64 token rows (33-48 and 49-64 nodes) in float32 and bf16
    "f32-40-nodes": ("f32", 4, 4, 64, [[-1] + [j // 2 for j in range(0, 39)]], [100]),
    "f32-61-nodes": ("f32", 4, 4, 64, [[-1] + [max(0, j - 3) for j in range(1, 61)]], [77]),
    "bf16-56-nodes": ("bf16", 4, 2, 128, [[-1] + [j // 3 for j in range(0, 55)]], [64]),
    # ragged batches on the register path (flat partition of each head's KV tiles)
    # (the cache capacity covers the longest prefix plus the largest tree, as the ABI requires)
    "f32-ragged": ("f32", 4, 4, 64, [[-1, 0, 1], [-1] + list(range(0, 20)), [-1, 0, 0, 0, 1]], [300, 1000, 17]),
    "bf16-ragged-mha": ("bf16", 4, 4, 128, [[-1, 0, 1, 1], [-1] + list(range(0, 9)), [-1], [-1, 0, 0, 2, 3, 3]],
                        [900, 3000, 40, 250]),
}


@pytest.mark.timeout(300)
@pytest.mark.parametrize("name", list(EDGE))
def test_edge_case_parity(rt, name):
    dtype, hq, hkv, d, parents, kv = EDGE[name]
    depth = max(8, max(_depth(p) for p in parents))
    shp = _edge_shape(dtype, hq, hkv, d, depth=depth)
    w = synth.custom(shp, parents, kv, seed=101, poison_tail=True)
    w.shape = synth.Shape("edge", dtype, hq * d, hq, hkv, d, shp.vocab, len(parents),
                          max(len(p) for p in parents), depth, 8)
    _say(f"[edge {name}] building")
    case = workload.finish(w)
    _say(f"[edge {name}] running GPU step")
    compare(case, rt.run(case.w, x_out=True, tok_rank=True), f"edge {name}")


# Vocabulary sizes that take each form of the vocabulary pass: one wave per row
# (<= 64 tiles of 64 tokens), four waves with 2, 8 and 16 tile keys per thread,
# and rows read whole (more than 4096 tiles).  "clustered" gives 24
# consecutive tokens (across a tile boundary) near-copies of one LM-head row
# scaled by 6-7.2, so that on many rows most of the top-k sits in one tile;
# "tied" gives 200 tokens one identical LM-head row (3x row 7) and token 5 the
# row 3.5x row 7, so that on many rows the top-k is token 5 followed by equal
# logits (more of them reach the candidate threshold than the sorted path takes).
VOCAB_TIERS = [
    (3001, 8, "plain"),        # a vocabulary that is not a multiple of 4 (unaligned logit rows)
    (3000, 16, "clustered"),
    (3000, 8, "tied"),
    (30000, 8, "clustered"),
    (30000, 16, "tied"),
    (70000, 8, "plain"),
    (40001, 8, "plain"),       # 256-row vocabulary tiles with a ragged last tile and unaligned logit rows
    (200000, 16, "clustered"),
    (300000, 8, "clustered"),
]


# 65-128 token rows take the LM head's 128 x 128 GEMM tile: two sequences of
# 60 and 40 nodes over a vocabulary that is a multiple of neither 4 nor 128.
@pytest.mark.timeout(300)
def test_gemm_128_row_tile(rt):
    vocab = 3001
    parents = [[-1] + [(j - 1) // 3 for j in range(1, 60)], [-1] + [max(0, j - 2) for j in range(1, 40)]]
    depth = max(8, max(_depth(p) for p in parents))
    shp = synth.Shape("edge", "bf16", 4 * 64, 4, 2, 64, vocab, 2, 60, depth, 8)
    # (the longest prefix goes with the largest tree: the cache holds max prefix + max nodes rows)
    w = synth.custom(shp, parents, [260, 90], seed=241, poison_tail=True)
    _say("[gemm 128-row tile, 100 rows] building")
    case = workload.finish(w)
    _say("[gemm 128-row tile, 100 rows] running GPU step")
    compare(case, rt.run(case.w, x_out=True, tok_rank=True), "gemm 128-row tile")


# At most 64 token rows over a vocabulary of more than two 64-row tiles per CU
# take the LM head's 64 x 256 tile: one row (every other x row a clamped copy),
# a partial tile and a full one, over a vocabulary that is a multiple of neither
# 4 nor 256 (unaligned logit rows, a ragged last tile).
@pytest.mark.timeout(300)
@pytest.mark.parametrize("n_nodes", [1, 33, 64])
def test_wide_vocab_token_rows(rt, n_nodes):
    vocab = 33001
    parents = [[-1] + [(j - 1) // 2 for j in range(1, n_nodes)]]
    depth = max(8, _depth(parents[0]))
    shp = synth.Shape("edge", "bf16", 4 * 64, 4, 2, 64, vocab, 1, n_nodes, depth, 8)
    w = synth.custom(shp, parents, [150], seed=233 + n_nodes, poison_tail=True)
    _say(f"[wide vocab {vocab}, {n_nodes} rows] building")
    case = workload.finish(w)
    _say(f"[wide vocab {vocab}, {n_nodes} rows] running GPU step")
    compare(case, rt.run(case.w, x_out=True, tok_rank=True), f"wide vocab {n_nodes} rows")


@pytest.mark.timeout(300)
@pytest.mark.parametrize("vocab,topk_out,mode", VOCAB_TIERS)
def test_vocab_tier_parity(rt, vocab, topk_out, mode):
    parents = [[-1, 0, 1, 1, 3, 0], [-1, 0, 0, 2]]
    shp = synth.Shape("edge", "bf16", 4 * 64, 4, 1, 64, vocab, 2, 6, 8, topk_out)
    w = synth.custom(shp, parents, [70, 40], seed=211, poison_tail=True)
    if mode != "plain":
        W = synth.bf16_bits_to_f32(w.lm_head).reshape(vocab, -1).copy()
        if mode == "clustered":
            c0 = 64 * 5 + 48
            for k in range(24):
                W[c0 + k] = W[7] * (6.0 + 0.05 * k) + 0.002 * W[100 + k]
        else:
            W[64:264] = W[7] * 3.0
            W[5] = W[7] * 3.5
        w.lm_head = synth.f32_to_bf16_bits(W).reshape(w.lm_head.shape)
    w.params = synth.AcceptParams(topk=topk_out, tau=1.0, min_lookahead=1, max_relaxed=2)
    _say(f"[vocab {vocab} k={topk_out} {mode}] building")
    case = workload.finish(w)
    _say(f"[vocab {vocab} k={topk_out} {mode}] running GPU step")
    compare(case, rt.run(case.w, tok_rank=True), f"vocab {vocab}")


# The LM head's GEMM form (bf16, more than 128 token rows in all): 256-row token
# tiles with rows past M, a vocabulary that is not a multiple of 4 (the logit
# rows are unaligned: scalar stores) nor of the 128-row vocabulary tile, and
# (300 nodes) a second token tile.
GEMM_CASES = {
    "218-nodes": [[-1] + [(j - 1) // 3 for j in range(1, 128)], [-1] + [(j - 1) // 2 for j in range(1, 90)]],
    "300-nodes": [[-1] + [(j - 1) // 3 for j in range(1, 128)], [-1] + [(j - 1) // 2 for j in range(1, 100)],
                  [-1] + [j - 1 for j in range(1, 60)], [-1] + [0] * 12],
}


@pytest.mark.timeout(300)
@pytest.mark.parametrize("name", list(GEMM_CASES))
def test_gemm_lm_head_parity(rt, name):
    parents = GEMM_CASES[name]
    depth = max(8, max(_depth(p) for p in parents))
    shp = synth.Shape("edge", "bf16", 4 * 64, 4, 2, 64, 3001, len(parents), max(len(p) for p in parents), depth, 8)
    # (the cache capacity covers the longest prefix plus the largest tree: the 128-node tree has the longest)
    w = synth.custom(shp, parents, [300, 90, 150, 20][:len(parents)], seed=505, poison_tail=True)
    assert int(w.node_off[-1]) > 128
    _say(f"[gemm {name}] building")
    case = workload.finish(w)
    _say(f"[gemm {name}] running GPU step")
    compare(case, rt.run(case.w, x_out=True, tok_rank=True), f"gemm {name}")


def _depth(parent):
    d = [0] * len(parent)
    for j in range(1, len(parent)):
        d[j] = d[parent[j]] + 1
    return max(d)


@pytest.mark.timeout(300)
@pytest.mark.parametrize("topk,tau,m,phi", [
    (1, 3.0, 2, 2), (8, 0.0, 2, 2), (8, 0.5, 1, 3), (8, 1.0, 0, 1), (8, 5.0, 3, 3), (4, 3.0, 0, 0),
    (16, 2.0, 1, 2),
])
def test_accept_parameter_sweep(rt, topk, tau, m, phi):
    params = synth.AcceptParams(topk=topk, tau=tau, min_lookahead=m, max_relaxed=phi)
    for cfg in (0,):
        w = synth.generate(cfg, params=params, poison_tail=True)
        if topk > 8:
            w.shape = synth.Shape(w.shape.name, w.shape.dtype, w.shape.hidden, w.shape.n_q_heads,
                                  w.shape.n_kv_heads, w.shape.head_dim, w.shape.vocab, w.shape.batch,
                                  w.shape.max_nodes, w.shape.max_depth, 16)
        _say(f"[sweep cfg{cfg} k={topk} tau={tau} m={m} phi={phi}] building")
        case = workload.finish(w)
        compare(case, rt.run(case.w), f"sweep k={topk} tau={tau} m={m} phi={phi}")


def test_stop_after_stages(rt):
    from paper_2511_01282_amd import binding
    case = workload.build(0)
    _say("[stop_after] attention only")
    out = rt.run(case.w, stop_after=binding.STOP_ATTN)
    np.testing.assert_allclose(out["attn_out"], case.attn, rtol=1e-4, atol=1e-4)
    _say("[stop_after] through logits")
    out = rt.run(case.w, stop_after=binding.STOP_LOGITS)
    np.testing.assert_allclose(out["logits"], case.z, rtol=1e-4, atol=1e-4)


@pytest.mark.timeout(300)
@pytest.mark.parametrize("cfg", [0, 1])
def test_stop_after_statistics(rt, cfg):
    # statistics and predicates only: the same values as the whole step, flags without
    # ON_PATH, and no path reduction (its outputs keep what they held)
    from paper_2511_01282_amd import binding
    case = workload.build(cfg)
    e = case.expected
    _say(f"[stop_after] statistics, config {cfg}")
    out = rt.run(case.w, stop_after=binding.STOP_STATS, tok_rank=True, x_out=True)
    for k in ("max_logit", "lse", "entropy", "topk_logprob"):
        np.testing.assert_allclose(out[k], e[k], rtol=RTOL, atol=ATOL, err_msg=k)
    np.testing.assert_array_equal(out["argmax"], e["argmax"])
    np.testing.assert_array_equal(out["flags"], e["flags"] & np.uint8(15))
    check_x(case, out["x_out"], f"stats {cfg}")
    check_rank(case, out["tok_rank"], out["logits"], f"stats {cfg}")


@pytest.mark.timeout(300)
def test_repeated_steps_are_bitwise_identical(rt):
    case = workload.build(1)
    plan = rt.make_plan(case.w)
    inputs = rt.upload(case.w)
    _say("[repeat] three runs on one plan/workspace")
    outs = [rt.run(case.w, plan=plan, inputs=inputs, repeat=r) for r in (1, 2, 3)]
    for o in outs[1:]:
        for k, v in o.items():
            if v is not None:
                np.testing.assert_array_equal(v, outs[0][k], err_msg=k)
    compare(case, outs[-1], "repeat")


def _wide_batch(n_seq=70, seed=401):
    """n_seq small ragged trees (1-7 nodes, prefixes of 0-150 rows): a batch past 64 sequences."""
    u = synth.uniform_stream(seed, 90, 0, 4 * n_seq + 200)
    parents, kv = [], []
    for s in range(n_seq):
        n = 1 + int(u[s] * 7)
        parents.append([-1] + [int(u[n_seq + s * 3 + k % 3] * k) for k in range(1, n)])
        kv.append(int(u[3 * n_seq + s] * 151))
    # the cache holds the longest prefix plus the largest tree: give the longest prefix a 7-node tree
    longest = int(np.argmax(kv))
    parents[longest] = [-1, 0, 1, 1, 3, 0, 5]
    return parents, kv


@pytest.mark.timeout(300)
def test_wide_batch_parity(rt):
    # 70 sequences: the register-path attention with per-sequence splits, the vocabulary
    # pass's node-offset scan over several groups of 64; sequence 13 has a malformed tree
    parents, kv = _wide_batch()
    parents[13] = [-1, 0, 2]                 # node 2 is its own parent
    shp = synth.Shape("edge", "bf16", 4 * 64, 4, 2, 64, 3000, len(parents), 7, 8, 8)
    w = synth.custom(shp, parents, kv, seed=402, poison_tail=True)
    _say("[wide batch] building 70 sequences")
    case = workload.finish(w)
    assert case.expected["seq_status"][13] == 5 and (case.expected["seq_status"] == 0).sum() == 69
    _say("[wide batch] running GPU step")
    compare(case, rt.run(case.w, x_out=True, tok_rank=True), "wide batch")


@pytest.mark.timeout(300)
def test_wide_batch_with_broken_node_offsets(rt):
    # one empty node range among 70: the offsets no longer describe the batch, so every
    # sequence is reported as a malformed tree (and nothing reads outside the buffers)
    parents, kv = _wide_batch(seed=403)
    shp = synth.Shape("edge", "bf16", 4 * 64, 4, 2, 64, 3000, len(parents), 7, 8, 8)
    w = synth.custom(shp, parents, kv, seed=404, poison_tail=True)
    case = workload.finish(w)
    bad = case.w
    w = synth.custom(shp, parents, kv, seed=404, poison_tail=True)
    bad.node_off = bad.node_off.copy()
    bad.node_off[40] = bad.node_off[41]      # sequence 40 empty, sequence 39 longer
    _say("[wide batch] running GPU step with an empty node range")
    # (the host arguments describe the real batch; only the device offsets are broken)
    out = rt.run(bad, step_kw=dict(max_nodes_in_batch=int(np.diff(w.node_off).max())))
    assert (out["seq_status"] == 5).all()
    assert (out["acc_len"] == -1).all() and (out["path"] == -1).all()
    assert (out["winner_leaf"] == -1).all() and (out["bonus"] == -1).all()


def test_invalid_device_data_is_reported_per_sequence(rt):
    shp = _edge_shape("bf16", 4, 2, 128)
    parents = [[-1, 0, 1], [-1, 0, 0], [-1, 0, 1], [-1, 0, 1], [-1, 0, 1]]
    w = synth.custom(shp, parents, [10, 10, 10, 10, 10], seed=7)
    w.shape = synth.Shape("edge", "bf16", 512, 4, 2, 128, shp.vocab, 5, 3, 8, 8)
    case = workload.finish(w)
    bad = case.w
    bad.parent = bad.parent.copy()
    bad.token = bad.token.copy()
    bad.src = bad.src.copy()
    bad.kv_len = bad.kv_len.copy()
    bad.parent[3 + 2] = 2          # seq 1: node 2 is its own parent
    bad.token[6 + 1] = shp.vocab   # seq 2: token out of range
    bad.src[9 + 2] = 3             # seq 3: unknown source tag
    bad.kv_len[4] = 10 ** 6        # seq 4: prefix longer than the cache
    _say("[invalid] running GPU step with malformed sequences 1-4")
    out = rt.run(bad, step_kw=dict(max_kv_len_in_batch=10))
    assert out["seq_status"].tolist() == [0, 5, 9, 9, 6]
    assert out["acc_len"].tolist()[1:] == [-1, -1, -1, -1]
    assert (out["path"][1:] == -1).all()
    assert out["acc_len"][0] == case.expected["acc_len"][0]
    assert out["path"][0].tolist() == case.expected["path"][0].tolist()
