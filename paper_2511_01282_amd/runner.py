"""Upload a verification workload to the GPU and run steps through the C ABI.

A workload is any object with the fields of ``respec_synth.Workload`` (numpy
arrays: hidden, k_cache, v_cache, lm_head, parent, node_off, kv_len, src,
token; a ``shape`` with the model sizes; accept ``params``).  bf16 tensors are
uint16 bit patterns on the host and ``torch.bfloat16`` on the device.
"""
from __future__ import annotations

import numpy as np
import torch

from . import binding


def _dev(a: np.ndarray, device, bf16: bool = False) -> torch.Tensor:
    a = np.ascontiguousarray(a)
    if bf16:
        return torch.from_numpy(a.view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(a).to(device)


def upload(w, device="cuda") -> dict:
    bf16 = w.shape.dtype == "bf16"
    return {
        "node_off": _dev(w.node_off.astype(np.int32), device),
        "kv_len": _dev(w.kv_len.astype(np.int32), device),
        "hidden": _dev(w.hidden, device, bf16),
        "k_cache": _dev(w.k_cache, device, bf16),
        "v_cache": _dev(w.v_cache, device, bf16),
        "lm_head": _dev(w.lm_head, device, bf16),
        "parent": _dev(w.parent.astype(np.int32), device),
        "token": _dev(w.token.astype(np.int32), device),
        "src": _dev(w.src.astype(np.uint8), device),
    }


def make_plan(w, device="cuda", *, max_batch=None, max_nodes=None, max_kv_len=None) -> binding.Plan:
    s = w.shape
    n_per = np.diff(w.node_off)
    return binding.Plan(
        hidden=s.hidden, n_q_heads=s.n_q_heads, n_kv_heads=s.n_kv_heads, head_dim=s.head_dim,
        vocab=s.vocab, dtype=binding.BF16 if s.dtype == "bf16" else binding.F32,
        max_batch=max_batch or max(1, len(n_per)),
        max_nodes=max_nodes or max(int(n_per.max()) if len(n_per) else 1, 1),
        max_depth=s.max_depth, max_kv_len=max_kv_len or max(int(w.kv_len.max()) if len(w.kv_len) else 0, 0),
        topk_out=s.topk_out, device=device)


def step_kwargs(w, params=None) -> dict:
    p = w.params if params is None else params
    n_per = np.diff(w.node_off)
    return dict(batch=len(n_per), total_nodes=int(w.node_off[-1]),
                max_nodes_in_batch=max(int(n_per.max()) if len(n_per) else 1, 1),
                max_kv_len_in_batch=int(w.kv_len.max()) if len(w.kv_len) else 0,
                kv_capacity=int(w.k_cache.shape[2]),
                topk=p.topk, tau=p.tau, min_lookahead=p.min_lookahead, max_relaxed=p.max_relaxed,
                stochastic=getattr(p, "stochastic", 0), temperature=getattr(p, "temperature", 1.0))


def run(w, *, plan=None, inputs=None, params=None, stop_after=binding.STOP_ALL, attn_out=True,
        device="cuda", repeat=1, step_kw=None, x_out=False, tok_rank=False) -> dict:
    """One (or ``repeat``) steps; returns every output as numpy arrays.

    ``step_kw`` overrides the host-side step arguments derived from ``w``; ``x_out`` and
    ``tok_rank`` also request the residual x (as the workload's bit patterns: uint16 for
    bf16) and the draft tokens' exact ranks.
    """
    kw = step_kwargs(w, params)
    kw.update(step_kw or {})
    plan = plan or make_plan(w, device, max_kv_len=kw["max_kv_len_in_batch"])
    inputs = inputs or upload(w, device)
    s = w.shape
    xd = (torch.bfloat16 if s.dtype == "bf16" else torch.float32) if x_out else None
    out = binding.alloc_outputs(total_nodes=kw["total_nodes"], batch=kw["batch"], hidden=s.hidden,
                                vocab=s.vocab, topk_out=s.topk_out, max_depth=s.max_depth, device=device,
                                attn_out=attn_out, x_dtype=xd, tok_rank=tok_rank)
    for _ in range(repeat):
        plan.step(inputs, out, stop_after=stop_after, **kw)
    torch.cuda.synchronize(device)
    res = {}
    for k, v in out.items():
        if v is None:
            res[k] = None
        elif v.dtype == torch.bfloat16:
            res[k] = v.view(torch.int16).cpu().numpy().view(np.uint16)
        else:
            res[k] = v.cpu().numpy()
    return res
