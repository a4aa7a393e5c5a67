"""A token-conditioned proxy target for decoding loops (test harness).

The verification step's one-layer proxy takes hidden states and K/V rows as
inputs.  Here they are looked up per token from seeded tables, so that a
context and a draft tree fully determine a step: the hidden state of a node
is E_h[token], the K/V rows of a token are E_k[token] and E_v[token] viewed as
heads, the prefix holds the rows of every context token but the last, and the
tree's rows follow it (the root is the context's last token).  With no
positional encoding the logits of a node depend only on the set of rows it
sees, so a node's distribution equals the one plain autoregressive decoding
sees after the same tokens.

The loop drives a drafting session (the library's or the oracle's) and a
verification function (the GPU path or the oracle), and returns the context.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

import respec_synth as synth

_TABLE_STREAMS = {"E_h": 21, "E_k": 22, "E_v": 23, "W": 24}


@dataclass
class LoopModel:
    shape: synth.Shape
    params: synth.AcceptParams
    E_h: np.ndarray   # [V][Hd]
    E_k: np.ndarray   # [V][Hkv*D]
    E_v: np.ndarray   # [V][Hkv*D]
    W: np.ndarray     # [V][Hd]
    seed: int


def make_model(seed=11, *, vocab=512, hidden=256, n_heads=4, head_dim=64, w_std=0.5, max_depth=32, max_nodes=64,
               params=None) -> LoopModel:
    shape = synth.Shape("loop", "f32", hidden, n_heads, n_heads, head_dim, vocab, 1, max_nodes, max_depth, 8)
    kvw = n_heads * head_dim

    def table(name, cols, std):
        return (synth.normal_stream(seed, _TABLE_STREAMS[name], 0, vocab * cols) * std).astype(
            np.float32).reshape(vocab, cols)

    return LoopModel(shape, params or synth.AcceptParams(), table("E_h", hidden, 1.0), table("E_k", kvw, 1.0),
                     table("E_v", kvw, 1.0), table("W", hidden, w_std), seed)


def workload(m: LoopModel, text, parent, token, src) -> synth.Workload:
    """One verification step of tree (parent, token, src) after context ``text``."""
    s = m.shape
    text = np.asarray(text, np.int32)
    token = np.asarray(token, np.int32)
    L, N = len(text) - 1, len(parent)
    Hkv, D = s.n_kv_heads, s.head_dim
    rows = np.concatenate([text[:-1], token])                 # prefix rows, then the tree's
    k = m.E_k[rows].reshape(L + N, Hkv, D).transpose(1, 0, 2)[None].copy()
    v = m.E_v[rows].reshape(L + N, Hkv, D).transpose(1, 0, 2)[None].copy()
    return synth.Workload(s, m.seed, m.E_h[token].copy(), np.ascontiguousarray(k), np.ascontiguousarray(v), m.W,
                          np.asarray(parent, np.int32), np.array([0, N], np.int32), np.array([L], np.int32),
                          np.asarray(src, np.uint8), token, m.params, {"kind": "loop"})


def prompt(seed=5, n=48, vocab=512, repeat=(8, 20, 30)):
    """A synthetic prompt with one copied span (so retrieval has something to find)."""
    t = np.minimum((synth.uniform_stream(seed, 31, 0, n) * vocab).astype(np.int64), vocab - 1).astype(np.int32)
    a, b, c = repeat
    t[c:c + (b - a)] = t[a:b]
    return t


def greedy_decode(m: LoopModel, prompt_tokens, n_tokens, verify):
    """Plain autoregressive greedy decoding: one root-only tree per token."""
    text = list(int(x) for x in prompt_tokens)
    for _ in range(n_tokens):
        out = verify(workload(m, text, [-1], [text[-1]], [0]))
        text.append(int(out["bonus"][0]))
    return text


def speculative_decode(m: LoopModel, session, prompt_tokens, n_steps, verify, log=None):
    """Algorithm 1's loop: propose (trigger, retrieval, tree) -> verify -> commit.

    ``session`` has append(tokens, entropy), propose() -> (parent, token, src,
    retrieved), commit(token, path, acc_len, bonus, entropy) and text().
    Returns the context and the per-step (retrieved, n_nodes, acc_len).
    """
    session.append(prompt_tokens, None)
    steps = []
    for _ in range(n_steps):
        parent, token, src, retrieved = session.propose()
        text = session.text()
        out = verify(workload(m, text, parent, token, src))
        acc = int(out["acc_len"][0])
        session.commit(token, out["path"][0], acc, int(out["bonus"][0]), out["entropy"])
        steps.append((bool(retrieved), len(parent), acc))
        if log is not None:
            log(steps[-1])
    return session.text(), steps
