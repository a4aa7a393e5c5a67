#!/usr/bin/env python3
"""Tree-verification throughput on one MI355X.

One step = one pass of the whole hot path (tree-masked attention + residual,
LM head, fused vocab pass with strict/relaxed acceptance, path reduction)
over one batch of synthetic input, through the C ABI.  Default workload: the
7B-shaped verify (hidden 4096, 32/32 heads, head_dim 128, vocab 32000, KV
length 2048, a 26-node random draft tree, bf16 with fp32 accumulation).

Inputs are resident in HBM before timing starts.  Several copies of the large
inputs (K/V cache, LM head, hidden states) are rotated from step to step so
that the working set exceeds the 256 MB Infinity Cache and every step streams
its bytes from HBM.  The timed region runs K plain steps.  A second pass of K
steps records HIP events on the step's stream around each stage (attention
with its split merge, LM head, vocabulary pass); they give each stage's
average duration for the roofline figures, reported against the vendor peaks
and against ceilings measured in the same run (a plain streaming read and a
matrix-core loop).  The CPU baseline times the oracle on the host cores on a
bounded sample of whole steps of the same workload (and on one thread for the
two smallest workloads); its result also checks the timed step's decisions.

Prints ONE JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0    # dense MFMA bf16
FP32_PEAK_TFLOPS = 157.3
MALL_BYTES = 256 << 20


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def stage_bytes(w, M, es):
    """Algorithmic HBM bytes per launch of each stage (inputs read once, outputs written once)."""
    s = w.shape
    kv_rows = sum(int(w.kv_len[b]) + int(w.node_off[b + 1] - w.node_off[b]) for b in range(len(w.kv_len)))
    attn = 2 * s.n_kv_heads * kv_rows * s.head_dim * es + 2 * M * s.hidden * es   # K,V + h in + x out
    lm = s.vocab * s.hidden * es + M * s.hidden * es + M * s.vocab * 4            # W + x + logits out
    # the LM-head epilogue reduces every 64-logit tile of a row to 16 bytes of statistics
    # (m, S, T, argmax); the vocabulary pass reads those, re-reads the K tiles per wave
    # whose maxima can hold the row's top-K (at least K = 8 or 16 tiles of 256 bytes per
    # wave, four waves per row past 64 tiles), and reads one logit per child
    n_vtiles = (s.vocab + 63) // 64
    ko = 8 if s.topk_out <= 8 else 16
    wpr = 4 if n_vtiles > 64 else 1
    vocab = M * n_vtiles * 16 + M * wpr * ko * 256 + M * 4
    vis = 0
    for b in range(len(w.kv_len)):
        lo, hi = int(w.node_off[b]), int(w.node_off[b + 1])
        depth = [0] * (hi - lo)
        for j in range(1, hi - lo):
            depth[j] = depth[int(w.parent[lo + j])] + 1
        vis += sum(int(w.kv_len[b]) + d + 1 for d in depth)
    attn_flops = 4 * s.n_q_heads * s.head_dim * vis                                # QK^T + PV
    lm_flops = 2 * M * s.vocab * s.hidden
    return dict(attn=attn, lm=lm, vocab=vocab, attn_flops=attn_flops, lm_flops=lm_flops)


STAGE_SOURCES = {"attention": ("attention.hip", "AttnArgs"), "lm_head": ("lmhead.hip", "LmArgs"),
                 "vocab_pass": ("vocab.hip", "VocabArgs")}


def stage_source_hash(stage):
    """Hash of what a stage's kernels are compiled from: its .hip file, common.hpp and its
    argument struct in kernels.hpp (the other declarations there do not change it)."""
    import hashlib
    src, struct = STAGE_SOURCES[stage]
    csrc = os.path.join(ROOT, "paper_2511_01282_amd", "csrc")
    h = hashlib.sha256()
    for f in (src, "common.hpp"):
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(fh.read())
    text = open(os.path.join(csrc, "kernels.hpp")).read()
    a = text.index("struct %s {" % struct)
    h.update(text[a:text.index("};", a) + 2].encode())
    return h.hexdigest()[:16]


def stage_traffic(shape_name, stage):
    """HBM bytes per launch of a stage's kernels from the committed counter profile of the
    workload (FETCH_SIZE and WRITE_SIZE, calibrated), or None when there is none or the
    stage's sources changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", "verify_step_%s_hbm_traffic.txt" % shape_name.replace("-", "_"))
    if not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        parts = line.split()
        if len(parts) == 3 and parts[0] in ("traffic_bytes", "source_sha256_16") and parts[1] == stage:
            fields[parts[0]] = parts[2]
    if "traffic_bytes" not in fields or fields.get("source_sha256_16") != stage_source_hash(stage):
        return None
    return int(fields["traffic_bytes"])


def draft_host_timing(seconds=1.0):
    """Host cost of the drafting side of a step (trigger, suffix-automaton retrieval, EMA
    selection, BuildDraftTree, then feedback and context append), library against oracle.

    Scenario (copy-heavy, like summarisation or retrieval-augmented generation): a context
    of 8192 synthetic tokens (Zipf(1.1) over a 32000 vocabulary) and an output that copies
    the span starting at token 1000 with one token in ten replaced.  Every token's entropy
    is 0.5 nats, so the trigger fires.  Each round proposes a tree; the stand-in verifier
    accepts the tree's longest greedy match of the output, the bonus is the output's next
    token, and the round commits.  Only the library calls (propose, commit through the
    C ABI, buffers allocated once) and the oracle's propose and commit are timed; both run
    the same rounds, so their accepted lengths must agree.
    """
    import ctypes
    import numpy as np
    import respec_synth as synth
    from paper_2511_01282_amd import draft
    import oracle.draft as od

    n, V = 8192, 32000
    cdf = np.cumsum(np.arange(1, V + 1, dtype=np.float64) ** -1.1)
    cdf /= cdf[-1]
    ctx = np.searchsorted(cdf, synth.uniform_stream(9, 40, 0, n)).astype(np.int32)
    out = ctx[1000:1000 + 4000].copy()
    sub = synth.uniform_stream(9, 41, 0, len(out)) < 0.1
    out[sub] = np.searchsorted(cdf, synth.uniform_stream(9, 42, 0, len(out)))[sub]
    ent = np.full(n, 0.5, np.float32)

    def outcome(parent, token, pos):
        """Greedy match of the output along the tree: the accepted path and the bonus token."""
        kids = {}
        for j in range(1, len(parent)):
            kids.setdefault(int(parent[j]), []).append(j)
        path, v = [0], 0
        while pos + len(path) - 1 < len(out):
            nxt = [c for c in kids.get(v, []) if token[c] == out[pos + len(path) - 1]]
            if not nxt:
                break
            v = nxt[0]
            path.append(v)
        acc = len(path) - 1
        return path, acc, int(out[min(pos + acc, len(out) - 1)])

    L = draft.lib()
    sess = draft.DraftSession()
    sess.append(ctx, ent)
    cap = sess.params.tree.max_nodes
    parent, token = np.empty(cap, np.int32), np.empty(cap, np.int32)
    src, res = np.empty(cap, np.uint8), draft.DraftResult()
    path_buf = np.empty(cap, np.int32)
    node_ent = np.full(cap, 0.5, np.float32)
    h, pp, tp, sp = sess._h, parent.ctypes.data, token.ctypes.data, src.ctypes.data
    lib_acc, t_lib, pos = [], 0.0, 0
    while (t_lib < seconds / 2 or len(lib_acc) < 20) and pos < len(out) - 64:
        t0 = time.perf_counter()
        st = L.respec_draft_session_propose(h, pp, tp, sp, cap, ctypes.byref(res))
        t_lib += time.perf_counter() - t0
        m = res.n_nodes
        path, acc, bonus = outcome(parent[:m], token[:m], pos)
        path_buf[:acc + 1] = path
        t0 = time.perf_counter()
        st |= L.respec_draft_session_commit(h, tp, path_buf.ctypes.data, acc, bonus, node_ent.ctypes.data)
        t_lib += time.perf_counter() - t0
        if st:
            raise RuntimeError("drafting session call failed")
        lib_acc.append(acc)
        pos += acc + 1
    o = od.Session()
    o.append([int(v) for v in ctx], [float(v) for v in ent])
    or_acc, t_or, pos = [], 0.0, 0
    e_list = [0.5] * cap
    while len(or_acc) < len(lib_acc) and (t_or < seconds / 2 or len(or_acc) < 5):
        t0 = time.perf_counter()
        r = o.propose()
        t_or += time.perf_counter() - t0
        path, acc, bonus = outcome(r["parent"], r["token"], pos)
        t0 = time.perf_counter()
        o.commit(r["token"], path, acc, bonus, e_list)
        t_or += time.perf_counter() - t0
        or_acc.append(acc)
        pos += acc + 1
    return {"us_per_step": round(t_lib / len(lib_acc) * 1e6, 2), "rounds": len(lib_acc),
            "mean_accepted": round(float(np.mean(lib_acc)), 3), "context_tokens": n,
            "oracle_us_per_step": round(t_or / len(or_acc) * 1e6, 1), "oracle_rounds": len(or_acc),
            "oracle_agrees": or_acc == lib_acc[:len(or_acc)],
            "what": "propose (trigger, retrieval, selection, tree) + commit (EMA, append), host, 1 thread"}


def input_sha256(w):
    """SHA-256 over every input array of the step (after the draft tokens are set)."""
    import hashlib
    import numpy as np
    h = hashlib.sha256()
    for k in ("hidden", "k_cache", "v_cache", "lm_head", "parent", "token", "src", "node_off", "kv_len"):
        h.update(np.ascontiguousarray(getattr(w, k)).tobytes())
    return h.hexdigest()


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def time_oracle_steps(oracle, w, seconds, min_steps=3, max_single=30.0):
    """Whole oracle steps of w, timed one by one: at least min_steps (one if a step takes more
    than max_single seconds) and until `seconds` have passed.  Returns (times, last result)."""
    times, res = [], None
    while len(times) < min_steps or sum(times) < seconds:
        t1 = time.perf_counter()
        res = oracle.verify_step(w)
        times.append(time.perf_counter() - t1)
        if times[0] > max_single:
            break
    return times, res


def min_decision_margin(w, z):
    """Smallest distance of a decision from its threshold in logits z: each row's top-1/top-2
    gap, and each non-greedy draft token's distance from the tau and rank-k boundaries."""
    import numpy as np
    p = w.params
    z32 = np.asarray(z, np.float32)
    m = float("inf")
    for b in range(len(w.node_off) - 1):
        lo, hi = int(w.node_off[b]), int(w.node_off[b + 1])
        for i in range(lo, hi):
            t2 = np.partition(z32[i], -2)[-2:]
            m = min(m, float(t2[1]) - float(t2[0]))
        for j in range(lo + 1, hi):
            row, t = z32[lo + int(w.parent[j])], int(w.token[j])
            order = np.lexsort((np.arange(row.shape[0]), -row.astype(np.float64)))
            if t == int(order[0]):
                continue
            m = min(m, abs(float(row[order[0]]) - float(row[t]) - p.tau))
            r = int(np.nonzero(order == t)[0][0])
            if p.topk < row.shape[0]:
                m = min(m, float(row[t]) - float(row[order[p.topk]]) if r < p.topk
                        else float(row[order[p.topk - 1]]) - float(row[t]))
    return m


def probe_ceilings(dev, stream):
    """Measured ceilings: a plain 1 GiB streaming read (larger than the 256 MB MALL) and bf16
    matrix-core loops of both MFMA shapes; the best of 5 launches of each configuration."""
    import ctypes
    import torch
    from paper_2511_01282_amd import binding
    L = binding.lib()
    L.respec_probe_read.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int32, ctypes.c_int32,
                                    ctypes.c_void_p, ctypes.c_void_p]
    L.respec_probe_mfma.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                    ctypes.c_void_p]
    n = 1 << 30
    buf = torch.empty(n, dtype=torch.uint8, device=dev)
    sink = torch.empty(4096, dtype=torch.int32, device=dev)
    wgs, iters = 4096, 1000
    fsink = torch.empty(wgs * 256, dtype=torch.float32, device=dev)
    s = stream.cuda_stream

    def best(launch, count=5):
        ts = []
        for _ in range(count + 1):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            if launch() != 0:
                raise RuntimeError("probe launch failed")
            b.record(stream)
            b.synchronize()
            ts.append(a.elapsed_time(b) * 1e-3)
        return min(ts[1:])

    t_read = min(best(lambda: L.respec_probe_read(buf.data_ptr(), n, g, d, sink.data_ptr(), s))
                 for g, d in ((1024, 8), (4096, 8), (4096, 16)))
    tf = {}
    for shape, flops_each in ((0, 16384), (1, 32768)):
        t = best(lambda: L.respec_probe_mfma(wgs, iters, shape, fsink.data_ptr(), s))
        tf[shape] = wgs * 4 * iters * 8 * flops_each / t / 1e12
    return {"read_GBps": round(n / t_read / 1e9, 1), "mfma_bf16_TFLOPs": round(max(tf.values()), 1),
            "mfma_bf16_16x16x32_TFLOPs": round(tf[0], 1), "mfma_bf16_32x32x16_TFLOPs": round(tf[1], 1),
            "what": "1 GiB read once with 16-byte loads (best of 1024 or 4096 workgroups, 8 or 16 loads in "
                    "flight per thread); 4096 workgroups x 4 waves of 8 independent bf16 MFMA chains per shape; "
                    "best of 5 launches"}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", type=int, default=1, help="workload shape (default: 7B-shaped 26-node verify)")
    ap.add_argument("--rotate", type=int, default=0, help="input copies rotated per step (0: enough to exceed MALL)")
    ap.add_argument("--cpu-seconds", type=float, default=8.0, help="time budget of the CPU oracle sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-stochastic", action="store_true", help="skip the speculative-sampling pass")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="also run a plain device copy of this many MiB (counter calibration)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(the verification step of one tree runs on one device).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import respec_synth as synth
    from paper_2511_01282_amd import binding, runner

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    cfg = args.config
    shp = synth.CONFIGS[cfg]
    es = 2 if shp.dtype == "bf16" else 4
    log(f"[bench] generating workload {cfg} ({shp.name})")
    w = synth.generate(cfg)
    M = int(w.node_off[-1])
    B = len(w.kv_len)

    # ---- CPU baseline leg: the oracle on the host cores, whole steps of this workload ----
    # (its logits do not depend on the draft tokens, so its first step also gives the argmax
    # that the workload's argmax-prefix rule needs, and its decisions check the GPU's below)
    cpu, expected, prefix_from = None, None, "gpu argmax (no oracle run)"
    if not args.no_cpu_baseline:
        import oracle
        nproc = oracle.threads()
        log(f"[bench] timing the CPU oracle on the host ({nproc} threads)")
        times, res = time_oracle_steps(oracle, w, args.cpu_seconds)
        z = res["logits"]
        w.token = synth.apply_prefix_rule(w, np.argmax(z.astype(np.float32), axis=1).astype(np.int32))
        prefix_from = "oracle argmax"
        expected = oracle.decide(w, z)
        margin = min_decision_margin(w, z)
        one = {}
        for c in (0, 1):
            oracle.set_threads(1)
            wc = w if c == cfg else synth.generate(c)
            tc, _ = time_oracle_steps(oracle, wc, 0.0)
            one[f"C{c}"] = {"ms_per_step": round(float(np.median(tc)) * 1e3, 1), "runs": len(tc)}
            log(f"[bench] oracle on 1 thread, workload {c}: {one[f'C{c}']['ms_per_step']} ms/step")
        oracle.set_threads(nproc)
        med = float(np.median(times))
        cpu = {"value": round(1.0 / med, 4), "unit": "steps/s", "cores": nproc, "kind": "oracle",
               "sample": f"{len(times)} whole steps of the same workload (attention, LM head, vocab statistics, "
                         f"acceptance, path), float64, {sum(times):.1f} s; value = 1 / median step time",
               "ms_per_step_median": round(med * 1e3, 1), "ms_per_step_min": round(min(times) * 1e3, 1),
               "cpu_model": cpu_model(), "one_thread": one}

    plan = runner.make_plan(w, dev)
    base = runner.upload(w, dev)
    kw = runner.step_kwargs(w)
    out = binding.alloc_outputs(total_nodes=M, batch=B, hidden=shp.hidden, vocab=shp.vocab,
                                topk_out=shp.topk_out, max_depth=shp.max_depth, device=dev, attn_out=False)
    if expected is None:
        # draft tokens: the workload's argmax-prefix rule, using the GPU's own argmax
        plan.step(base, out, **kw)
        torch.cuda.synchronize()
        w.token = synth.apply_prefix_rule(w, out["argmax"].cpu().numpy())
        base["token"].copy_(torch.from_numpy(w.token.astype(np.int32)))
    sha = input_sha256(w)

    set_bytes = sum(base[k].numel() * base[k].element_size() for k in ("k_cache", "v_cache", "lm_head", "hidden"))
    R = args.rotate or max(2, math.ceil(4 * MALL_BYTES / set_bytes))
    sets = [base]
    for _ in range(R - 1):
        s = dict(base)
        for k in ("k_cache", "v_cache", "lm_head", "hidden"):
            s[k] = base[k].clone()
        sets.append(s)
    log(f"[bench] {R} rotated input sets of {set_bytes / 2**20:.1f} MiB")

    stream = torch.cuda.current_stream(dev)
    for i in range(args.warmup):
        plan.step(sets[i % R], out, stream=stream, **kw)
    torch.cuda.synchronize()

    K = args.steps
    # timed region: K plain steps (no per-stage events), bracketed by synchronisations
    torch.cuda.synchronize()
    log(f"[bench] timing {K} steps")
    t0 = time.perf_counter()
    for i in range(K):
        plan.step(sets[i % R], out, stream=stream, **kw)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = wall * 1e3 / K

    # the timed steps' outputs (every set holds the same inputs) against the oracle's decisions
    check = {"checked": False}
    if expected is not None:
        got = {k: out[k].cpu().numpy() for k in ("argmax", "flags", "path", "acc_len", "bonus", "winner_leaf",
                                                 "leaf_acc_len", "seq_status")}
        mism = {k: int((got[k] != expected[k]).sum()) for k in got}
        check = {"checked": True, "agrees": not any(mism.values()), "mismatches": mism,
                 "min_decision_margin": float(f"{margin:.3g}"), "acc_len": got["acc_len"].tolist(),
                 "what": "argmax, flags, path, acc_len, bonus, winner, per-leaf lengths and statuses of the last "
                         "timed step, bit for bit against the oracle (float64) on the same inputs"}
        log(f"[bench] self-check against the oracle: {'agrees' if check['agrees'] else mism}")

    # per-stage durations: a second pass of K steps with HIP events that the library
    # takes from the kernels' own dispatches (start of attention, end of the split
    # merge, of the LM head and of the vocabulary pass), on the step's stream
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(K)]
    for row in evs:
        for e in row:
            e.record(stream)
    torch.cuda.synchronize()
    for i in range(K):
        plan.step(sets[i % R], out, stream=stream, stage_events=evs[i], **kw)
    torch.cuda.synchronize()

    st = {"attn": [], "lm": [], "vocab": [], "step": []}
    for row in evs:
        st["attn"].append(row[0].elapsed_time(row[1]))
        st["lm"].append(row[1].elapsed_time(row[2]))
        st["vocab"].append(row[2].elapsed_time(row[3]))
        st["step"].append(row[0].elapsed_time(row[3]))
    avg = {k: float(np.mean(v)) for k, v in st.items()}
    nb = stage_bytes(w, M, es)
    stages = {
        "attention": {"us": avg["attn"] * 1e3, "GB/s": nb["attn"] / (avg["attn"] * 1e-3) / 1e9,
                      "TFLOP/s": nb["attn_flops"] / (avg["attn"] * 1e-3) / 1e12, "bytes": nb["attn"]},
        "lm_head": {"us": avg["lm"] * 1e3, "GB/s": nb["lm"] / (avg["lm"] * 1e-3) / 1e9,
                    "TFLOP/s": nb["lm_flops"] / (avg["lm"] * 1e-3) / 1e12, "bytes": nb["lm"]},
        "vocab_pass": {"us": avg["vocab"] * 1e3, "GB/s": nb["vocab"] / (avg["vocab"] * 1e-3) / 1e9,
                       "bytes": nb["vocab"]},
        "step_events_us": avg["step"] * 1e3,
        # distribution of the event-timed steps (attention start to vocabulary-pass end)
        "step_us_p10": float(np.percentile(st["step"], 10)) * 1e3,
        "step_us_p50": float(np.percentile(st["step"], 50)) * 1e3,
        "step_us_p90": float(np.percentile(st["step"], 90)) * 1e3,
    }
    stochastic = None
    if not args.no_stochastic:
        # stochastic verification (speculative sampling, Section 3.4 for drafter outputs) on the
        # same inputs: drafter distributions near the target's (softmax of the logits plus
        # N(0, 0.5^2) noise) and seeded uniforms, made before the timed region
        g = torch.Generator(device=dev)
        g.manual_seed(5)
        q = torch.softmax(out["logits"] + 0.5 * torch.randn(out["logits"].shape, generator=g, device=dev), dim=-1)
        q = q.contiguous()
        u = torch.rand((M, 2), generator=g, device=dev)
        out_s = binding.alloc_outputs(total_nodes=M, batch=B, hidden=shp.hidden, vocab=shp.vocab,
                                      topk_out=shp.topk_out, max_depth=shp.max_depth, device=dev, attn_out=False)
        sets_s = [dict(x, draft_prob=q, uniform=u) for x in sets]
        kw_s = dict(kw, stochastic=1, temperature=1.0)
        for i in range(max(2, args.warmup // 4)):
            plan.step(sets_s[i % R], out_s, stream=stream, **kw_s)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(K):
            plan.step(sets_s[i % R], out_s, stream=stream, **kw_s)
        torch.cuda.synchronize()
        wall_s = time.perf_counter() - t0
        evs_s = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(K)]
        for row in evs_s:
            for e in row:
                e.record(stream)
        torch.cuda.synchronize()
        for i in range(K):
            plan.step(sets_s[i % R], out_s, stream=stream, stage_events=evs_s[i], **kw_s)
        torch.cuda.synchronize()
        stochastic = {
            "steps_per_s": round(K / wall_s, 2), "us_per_step": round(wall_s * 1e6 / K, 2),
            "vocab_pass_us": round(float(np.mean([r[2].elapsed_time(r[3]) for r in evs_s])) * 1e3, 3),
            "mean_accepted": round(float(out_s["acc_len"].float().mean().item()), 3),
            "what": "same step with speculative-sampling verification (temperature 1); the vocabulary "
                    "stage includes the sampling walk",
        }
        log(f"[bench] stochastic: {stochastic['us_per_step']:.1f} us/step, vocab stage "
            f"{stochastic['vocab_pass_us']:.1f} us")

    ceil = probe_ceilings(dev, stream)
    log(f"[bench] measured ceilings: read {ceil['read_GBps']} GB/s, bf16 MFMA {ceil['mfma_bf16_TFLOPs']} TFLOP/s "
        f"(16x16x32: {ceil['mfma_bf16_16x16x32_TFLOPs']})")

    dom = max(("attention", "lm_head", "vocab_pass"), key=lambda k: stages[k]["us"])
    achieved = stages[dom]["GB/s"]
    traffic = stage_traffic(shp.name, dom)
    roofline = {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic}
    # every stage against the vendor peaks and the measured ceilings, with the targets
    # (>= 60 % of HBM for the attention and vocabulary passes, >= 50 % bf16 MFMA for the LM head)
    peak_tf = BF16_PEAK_TFLOPS if shp.dtype == "bf16" else FP32_PEAK_TFLOPS
    ai = nb["lm_flops"] / nb["lm"]
    attainable = min(peak_tf, ai * HBM_PEAK_GBS / 1e3)
    per_stage = {}
    for k in ("attention", "vocab_pass", "lm_head"):
        gbs = stages[k]["GB/s"]
        per_stage[k] = {"GB/s": round(gbs, 1), "frac_hbm_peak": round(gbs / HBM_PEAK_GBS, 4),
                        "frac_measured_read": round(gbs / ceil["read_GBps"], 4),
                        "bytes": int(stages[k]["bytes"]), "traffic": stage_traffic(shp.name, k)}
    per_stage["attention"]["target_frac_hbm"] = 0.6
    per_stage["vocab_pass"]["target_frac_hbm"] = 0.6
    tf = stages["lm_head"]["TFLOP/s"]
    per_stage["lm_head"].update({
        "TFLOP/s": round(tf, 1), "mfma_frac_peak": round(tf / peak_tf, 4),
        "mfma_frac_measured": round(tf / ceil["mfma_bf16_TFLOPs"], 4) if shp.dtype == "bf16" else None,
        "target_mfma_frac": 0.5, "arithmetic_intensity": round(ai, 1),
        "attainable_tflops": round(attainable, 1), "frac_of_attainable": round(tf / attainable, 4)})
    roofline["stages"] = per_stage
    roofline["measured_ceilings"] = ceil
    if dom == "lm_head":
        roofline["mfma_frac"] = per_stage["lm_head"]["mfma_frac_peak"]
        roofline["attainable_tflops"] = round(attainable, 1)
        roofline["frac_of_attainable"] = per_stage["lm_head"]["frac_of_attainable"]
    log(f"[bench] {ms_step * 1e3:.1f} us/step; stages " +
        ", ".join(f"{k} {stages[k]['us']:.1f} us" for k in ("attention", "lm_head", "vocab_pass")))

    if args.calib_copy_mib:
        # counter calibration: two plain kernels that each read and write exactly n bytes
        n = args.calib_copy_mib << 20
        a = torch.ones(n // 4, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        b.copy_(a)
        torch.mul(a, 2.0, out=b)
        torch.cuda.synchronize()

    draft_host = None if args.no_cpu_baseline else draft_host_timing()

    wl = {"workload": f"{shp.name}: {shp.dtype}, hidden {shp.hidden}, heads {shp.n_q_heads}/{shp.n_kv_heads}, "
                      f"head_dim {shp.head_dim}, vocab {shp.vocab}, batch {B}, nodes {M}, "
                      f"KV len {int(w.kv_len.max())}", "config_index": cfg, "rotated_input_sets": R,
          "input_sha256": sha, "draft_tokens": f"argmax-prefix rule from the {prefix_from}"}
    res = {
        "metric": "tree-verify steps/sec (attn+LM-head+accept), % of HBM and MFMA roofline",
        "value": round(K / wall, 2), "unit": "steps/s", "n_gpus": 1, "steps": K, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if shp.dtype == "bf16" else "f32", "data": "synthetic", "config": wl,
        "roofline": roofline, "cpu_baseline": cpu, "self_check": check, "draft_host": draft_host,
        "stochastic": stochastic,
        "stages": {k: ({kk: round(vv, 3) for kk, vv in v.items()} if isinstance(v, dict) else round(v, 3))
                   for k, v in stages.items()},
        "device": torch.cuda.get_device_name(dev),
    }
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
