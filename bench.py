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
average duration for the roofline figures.  The CPU baseline times the oracle
on the host cores on a bounded sample of the same workload.

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


def lmhead_source_hash():
    """Hash of what the LM-head kernel is compiled from: lmhead.hip, common.hpp and the
    LmArgs struct of kernels.hpp (the other launch declarations there do not change it)."""
    import hashlib
    csrc = os.path.join(ROOT, "paper_2511_01282_amd", "csrc")
    h = hashlib.sha256()
    for f in ("lmhead.hip", "common.hpp"):
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(fh.read())
    text = open(os.path.join(csrc, "kernels.hpp")).read()
    a = text.index("struct LmArgs {")
    h.update(text[a:text.index("};", a) + 2].encode())
    return h.hexdigest()[:16]


def lmhead_traffic(cfg):
    """HBM bytes per LM-head launch from the committed counter profile of the 7B-shaped
    workload, or None when the kernel sources changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", "lmhead_7b_26node_hbm_traffic.txt")
    if cfg != 1 or not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        parts = line.split()
        if len(parts) >= 2 and parts[0] in ("lmhead_traffic_bytes", "lmhead_source_sha256_16"):
            fields[parts[0]] = parts[1]
    if fields.get("lmhead_source_sha256_16") != lmhead_source_hash():
        return None
    return int(fields["lmhead_traffic_bytes"])


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


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", type=int, default=1, help="workload shape (default: 7B-shaped 26-node verify)")
    ap.add_argument("--rotate", type=int, default=0, help="input copies rotated per step (0: enough to exceed MALL)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="time budget of the CPU oracle sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="also run a plain device copy of this many MiB (counter calibration)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
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

    plan = runner.make_plan(w, dev)
    base = runner.upload(w, dev)
    kw = runner.step_kwargs(w)
    out = binding.alloc_outputs(total_nodes=M, batch=B, hidden=shp.hidden, vocab=shp.vocab,
                                topk_out=shp.topk_out, max_depth=shp.max_depth, device=dev, attn_out=False)

    # draft tokens: the workload's argmax-prefix rule, using the GPU's own argmax
    plan.step(base, out, **kw)
    torch.cuda.synchronize()
    argmax = out["argmax"].cpu().numpy()
    w.token = synth.apply_prefix_rule(w, argmax)
    base["token"].copy_(torch.from_numpy(w.token.astype(np.int32)))

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
    log(f"[bench] stochastic: {stochastic['us_per_step']:.1f} us/step, vocab stage {stochastic['vocab_pass_us']:.1f} us")

    dom = max(("attention", "lm_head", "vocab_pass"), key=lambda k: stages[k]["us"])
    achieved = stages[dom]["GB/s"]
    traffic = lmhead_traffic(cfg) if dom == "lm_head" else None
    roofline = {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic}
    if dom == "lm_head":
        # the matrix-core view of the same kernel: its fraction of the dense peak, and of the
        # attainable roofline min(peak, arithmetic intensity x HBM peak) at this token count
        peak_tf = BF16_PEAK_TFLOPS if shp.dtype == "bf16" else FP32_PEAK_TFLOPS
        ai = nb["lm_flops"] / nb["lm"]
        attainable = min(peak_tf, ai * HBM_PEAK_GBS / 1e3)
        roofline["mfma_frac"] = round(stages["lm_head"]["TFLOP/s"] / peak_tf, 4)
        roofline["attainable_tflops"] = round(attainable, 1)
        roofline["frac_of_attainable"] = round(stages["lm_head"]["TFLOP/s"] / attainable, 4)
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

    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        log("[bench] timing the CPU oracle on the host")
        n_done, t_cpu = 0, 0.0
        while t_cpu < args.cpu_seconds or n_done == 0:
            t1 = time.perf_counter()
            oracle.verify_step(w)
            t_cpu += time.perf_counter() - t1
            n_done += 1
        cpu = {"value": round(n_done / t_cpu, 4), "unit": "steps/s", "cores": oracle.threads(), "kind": "oracle",
               "sample": f"{n_done} full steps of the same workload (attention, LM head, vocab statistics, "
                         f"acceptance, path), float64, {t_cpu:.1f} s"}

    draft_host = None if args.no_cpu_baseline else draft_host_timing()

    wl = {"workload": f"{shp.name}: {shp.dtype}, hidden {shp.hidden}, heads {shp.n_q_heads}/{shp.n_kv_heads}, "
                      f"head_dim {shp.head_dim}, vocab {shp.vocab}, batch {B}, nodes {M}, "
                      f"KV len {int(w.kv_len.max())}", "config_index": cfg, "rotated_input_sets": R}
    res = {
        "metric": "tree-verify steps/sec (attn+LM-head+accept), % of HBM and MFMA roofline",
        "value": round(K / wall, 2), "unit": "steps/s", "n_gpus": 1, "steps": K, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if shp.dtype == "bf16" else "f32", "data": "synthetic", "config": wl,
        "roofline": roofline, "cpu_baseline": cpu, "draft_host": draft_host, "stochastic": stochastic,
        "stages": {k: ({kk: round(vv, 3) for kk, vv in v.items()} if isinstance(v, dict) else round(v, 3))
                   for k, v in stages.items()},
        "device": torch.cuda.get_device_name(dev),
    }
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
