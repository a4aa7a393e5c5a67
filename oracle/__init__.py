"""CPU oracle for one draft-tree verification step (TEST INFRASTRUCTURE ONLY).

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code with the GPU path:
the arithmetic lives in ``respec_oracle.c`` (plain C, float64), this file only
marshals numpy arrays and composes the steps in the paper's order:

  tree  -> tree-masked attention -> residual/rounding -> LM-head logits
        -> per-row statistics (entropy, Eq. 1) -> per-node strict/relaxed
           predicates (Section 3.4, Eq. 6-7) -> look-ahead tolerance per
           root-to-leaf chain and the winning path (Section 3.4, Algorithm 1).

Parity of the look-ahead step is unpinned beyond hand-worked cases: the
paper prints no worked example of it.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "respec_oracle.c")
_SO = os.path.join(_HERE, "librespec_oracle.so")
_LIB = None

F32, BF16 = 0, 1
FLAG_GREEDY, FLAG_TOPK, FLAG_TAU, FLAG_RELAXED, FLAG_ON_PATH = 1, 2, 4, 8, 16
SRC_RETRIEVED = 1


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (C11, OpenMP, no FP contraction)."""
    if force or not os.path.exists(_SO) or os.path.getmtime(_SO) < os.path.getmtime(_SRC):
        tmp = _SO + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-std=gnu11", "-O2", "-fopenmp", "-fPIC", "-shared",
                               "-ffp-contract=off", "-fno-fast-math", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _SO)
    return _SO


_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64


def _lib():
    global _LIB
    if _LIB is None:
        build()
        lib = ctypes.CDLL(_SO)
        sig = {
            "respec_oracle_tree": (_I32, [_P, _I32, _I32, _P, _P, _P]),
            "respec_oracle_attention": (None, [_I32, _P, _I32, _P, _P, _I32, _I32, _I32, _P,
                                               _I32, _I32, _I32, _P, _I32, _P]),
            "respec_oracle_residual": (None, [_I32, _P, _P, _I64, _P]),
            "respec_oracle_logits": (None, [_I32, _P, _I32, _I32, _P, _I32, _P]),
            "respec_oracle_row_stats": (None, [_P, _I32, _I32, _I32, _P, _P, _P, _P, _P, _P]),
            "respec_oracle_rank": (_I32, [_P, _I32, _I32]),
            "respec_oracle_node_flags": (None, [_I32, _P, _P, _P, _P, _I32, _P, _P, _I32,
                                                ctypes.c_float, _P, _P, _P]),
            "respec_oracle_lookahead": (_I32, [_I32, _P, _P, _I32, _I32]),
            "respec_oracle_threads": (_I32, []),
            "respec_oracle_set_threads": (None, [_I32]),
            "respec_oracle_path": (None, [_I32, _P, _P, _P, _P, _P, _I32, _I32, _I32, _P, _P,
                                          _P, _P, _P]),
            "respec_oracle_stoch_node": (_I32, [_I32, _P, ctypes.c_float, _P, _I32, _P, _P, _P,
                                                ctypes.c_float, _P]),
            "respec_oracle_stochastic": (_I32, [_I32, _P, _P, _P, _P, _I32, _P, _P, ctypes.c_float, _I32,
                                                _P, _P, _P, _P, _P, _P, _P, _P]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _LIB = lib
    return _LIB


def _c(a, dtype):
    a = np.ascontiguousarray(a, dtype=dtype)
    return a


def _p(a: np.ndarray) -> int:
    return a.ctypes.data


def _dt(w) -> int:
    return BF16 if w.shape.dtype == "bf16" else F32


# ---------------------------------------------------------------------------
# Stages
# ---------------------------------------------------------------------------

def threads() -> int:
    """OpenMP threads used by the oracle's parallel loops."""
    return int(_lib().respec_oracle_threads())


def set_threads(n: int) -> None:
    """Set the OpenMP threads of the oracle's parallel loops (timing on 1 thread or on all)."""
    _lib().respec_oracle_set_threads(int(n))


def tree(parent, max_depth: int):
    """(status, depth, anc[n][n], is_leaf) of one sequence's parent array."""
    parent = _c(parent, np.int32)
    n = parent.shape[0]
    depth = np.zeros(max(n, 1), np.int32)
    anc = np.zeros((max(n, 1), max(n, 1)), np.uint8)
    leaf = np.zeros(max(n, 1), np.uint8)
    st = _lib().respec_oracle_tree(_p(parent), n, max_depth, _p(depth), _p(anc), _p(leaf))
    return st, depth, anc, leaf


def attention(dtype: int, hidden, k_seq, v_seq, kv_len: int, anc, n_q_heads: int,
              n_kv_heads: int, head_dim: int, rows=None) -> np.ndarray:
    """Tree-masked attention of one sequence; hidden is [N][Hd], k/v [Hkv][cap][D]."""
    hidden = np.ascontiguousarray(hidden)
    k_seq = np.ascontiguousarray(k_seq)
    v_seq = np.ascontiguousarray(v_seq)
    anc = _c(anc, np.uint8)
    n_nodes, hd = hidden.shape
    rows = np.arange(n_nodes, dtype=np.int32) if rows is None else _c(rows, np.int32)
    out = np.zeros((rows.shape[0], hd), np.float64)
    _lib().respec_oracle_attention(dtype, _p(hidden), hd, _p(k_seq), _p(v_seq), k_seq.shape[1],
                                   kv_len, n_nodes, _p(anc), n_q_heads, n_kv_heads, head_dim,
                                   _p(rows), rows.shape[0], _p(out))
    return out


def residual(dtype: int, hidden, attn) -> np.ndarray:
    hidden = np.ascontiguousarray(hidden)
    attn = _c(attn, np.float64)
    x = np.zeros(attn.shape, np.float64)
    _lib().respec_oracle_residual(dtype, _p(hidden), _p(attn), attn.size, _p(x))
    return x


def logits(dtype: int, x, lm_head) -> np.ndarray:
    x = _c(x, np.float64)
    lm_head = np.ascontiguousarray(lm_head)
    n_rows, hd = x.shape
    vocab = lm_head.shape[0]
    z = np.zeros((n_rows, vocab), np.float64)
    _lib().respec_oracle_logits(dtype, _p(x), n_rows, hd, _p(lm_head), vocab, _p(z))
    return z


def row_stats(z32, topk_out: int) -> dict:
    z32 = _c(z32, np.float32)
    n, vocab = z32.shape
    out = dict(max_logit=np.zeros(n), argmax=np.zeros(n, np.int32), lse=np.zeros(n),
               entropy=np.zeros(n), topk_id=np.zeros((n, topk_out), np.int32),
               topk_logprob=np.zeros((n, topk_out)))
    _lib().respec_oracle_row_stats(_p(z32), n, vocab, topk_out, _p(out["max_logit"]),
                                   _p(out["argmax"]), _p(out["lse"]), _p(out["entropy"]),
                                   _p(out["topk_id"]), _p(out["topk_logprob"]))
    return out


def rank(row32, t: int) -> int:
    row32 = _c(row32, np.float32)
    return int(_lib().respec_oracle_rank(_p(row32), row32.shape[0], int(t)))


def node_flags(parent, token, src, z32, argmax, lse, topk: int, tau: float):
    parent = _c(parent, np.int32)
    token = _c(token, np.int32)
    src = _c(src, np.uint8)
    z32 = _c(z32, np.float32)
    argmax = _c(argmax, np.int32)
    lse = _c(lse, np.float64)
    n = parent.shape[0]
    flags = np.zeros(n, np.uint8)
    lp = np.zeros(n)
    rk = np.zeros(n, np.int32)
    _lib().respec_oracle_node_flags(n, _p(parent), _p(token), _p(src), _p(z32), z32.shape[1],
                                    _p(argmax), _p(lse), topk, float(tau), _p(flags), _p(lp), _p(rk))
    return flags, lp, rk


def lookahead(greedy, ok, m: int, phi: int) -> int:
    g = _c(greedy, np.uint8)
    o = _c(ok, np.uint8)
    if g.shape[0] == 0:
        g = np.zeros(1, np.uint8)
        o = np.zeros(1, np.uint8)
        return int(_lib().respec_oracle_lookahead(0, _p(g), _p(o), m, phi))
    return int(_lib().respec_oracle_lookahead(g.shape[0], _p(g), _p(o), m, phi))


def path(parent, is_leaf, depth, flags, argmax, max_depth: int, m: int, phi: int):
    """Winner of one validated tree; flags is updated in place with ON_PATH."""
    parent = _c(parent, np.int32)
    is_leaf = _c(is_leaf, np.uint8)
    depth = _c(depth, np.int32)
    argmax = _c(argmax, np.int32)
    assert flags.dtype == np.uint8 and flags.flags["C_CONTIGUOUS"]
    n = parent.shape[0]
    leaf_acc = np.zeros(n, np.int32)
    pth = np.zeros(max_depth + 1, np.int32)
    acc = np.zeros(1, np.int32)
    bonus = np.zeros(1, np.int32)
    wl = np.zeros(1, np.int32)
    _lib().respec_oracle_path(n, _p(parent), _p(is_leaf), _p(depth), _p(flags), _p(argmax),
                              max_depth, m, phi, _p(leaf_acc), _p(pth), _p(acc), _p(bonus), _p(wl))
    return dict(leaf_acc_len=leaf_acc, path=pth, acc_len=int(acc[0]), bonus=int(bonus[0]),
                winner_leaf=int(wl[0]))


def stoch_node(z_row, temperature: float, q_row, child_tok, child_model, u_acc, u_res: float):
    """One node of stochastic verification: (first accepted child index or -1, residual draw or -1)."""
    z = _c(z_row, np.float32)
    q = None if q_row is None else _c(q_row, np.float32)
    ct = _c(child_tok, np.int32) if len(child_tok) else np.zeros(1, np.int32)
    cm = _c(child_model, np.uint8) if len(child_model) else np.zeros(1, np.uint8)
    ua = _c(u_acc, np.float32) if len(u_acc) else np.zeros(1, np.float32)
    smp = np.zeros(1, np.int32)
    k = _lib().respec_oracle_stoch_node(z.shape[0], _p(z), float(temperature), None if q is None else _p(q),
                                        len(child_tok), _p(ct), _p(cm), _p(ua), float(u_res), _p(smp))
    return int(k), int(smp[0])


def stochastic(parent, token, src, z32, q, u, temperature: float, max_depth: int):
    """Stochastic verification of one sequence's tree (None for a malformed tree)."""
    parent = _c(parent, np.int32)
    token = _c(token, np.int32)
    src = _c(src, np.uint8)
    z32 = _c(z32, np.float32)
    q = None if q is None else _c(q, np.float32)
    u = _c(u, np.float32)
    n, V = z32.shape
    out = dict(first_acc=np.zeros(n, np.int32), sample=np.zeros(n, np.int32), acc_bit=np.zeros(n, np.uint8),
               path=np.zeros(max_depth + 1, np.int32), leaf_acc_len=np.zeros(n, np.int32))
    acc, bonus, wl = np.zeros(1, np.int32), np.zeros(1, np.int32), np.zeros(1, np.int32)
    st = _lib().respec_oracle_stochastic(n, _p(parent), _p(token), _p(src), _p(z32), V,
                                         None if q is None else _p(q), _p(u), float(temperature), max_depth,
                                         _p(out["first_acc"]), _p(out["sample"]), _p(out["acc_bit"]),
                                         _p(out["path"]), _p(acc), _p(bonus), _p(wl), _p(out["leaf_acc_len"]))
    if st != 0:
        return None
    out.update(acc_len=int(acc[0]), bonus=int(bonus[0]), winner_leaf=int(wl[0]))
    return out


# ---------------------------------------------------------------------------
# Whole step
# ---------------------------------------------------------------------------

# seq_status values for unusable sequences (the C ABI's status codes)
TREE_ERROR, CAPACITY_ERROR, TOKEN_ERROR = 5, 6, 9


def forward(w, rows_per_seq=None) -> dict:
    """Attention, residual and logits for every node (or the given local rows)."""
    shp = w.shape
    dt = _dt(w)
    B = len(w.node_off) - 1
    out = {"attn": [], "x": [], "z": [], "rows": []}
    for b in range(B):
        lo, hi = int(w.node_off[b]), int(w.node_off[b + 1])
        st, depth, anc, leaf = tree(w.parent[lo:hi], shp.max_depth)
        if st != 0:
            # malformed trees get a safe ancestor set: every node sees only itself
            anc = np.eye(hi - lo, dtype=np.uint8)
        rows = None if rows_per_seq is None else rows_per_seq[b]
        o = attention(dt, w.hidden[lo:hi], w.k_cache[b], w.v_cache[b], int(w.kv_len[b]), anc,
                      shp.n_q_heads, shp.n_kv_heads, shp.head_dim, rows)
        r = np.arange(hi - lo) if rows is None else np.asarray(rows)
        x = residual(dt, w.hidden[lo:hi][r], o)
        z = logits(dt, x, w.lm_head)
        out["attn"].append(o)
        out["x"].append(x)
        out["z"].append(z)
        out["rows"].append(r + lo)
    for k in ("attn", "x", "z", "rows"):
        out[k] = np.concatenate(out[k], axis=0)
    return out


def decide(w, z, params=None) -> dict:
    """Row statistics, predicates and accepted paths from full logits z [M][V]."""
    shp = w.shape
    p = w.params if params is None else params
    z32 = np.ascontiguousarray(z, dtype=np.float32)
    st = row_stats(z32, shp.topk_out)
    M = z32.shape[0]
    B = len(w.node_off) - 1
    flags = np.zeros(M, np.uint8)
    tok_lp = np.zeros(M)
    tok_rank = np.full(M, -1, np.int32)
    leaf_acc = np.full(M, -1, np.int32)
    paths = np.full((B, shp.max_depth + 1), -1, np.int32)
    acc_len = np.full(B, -1, np.int32)
    bonus = np.full(B, -1, np.int32)
    winner = np.full(B, -1, np.int32)
    status = np.zeros(B, np.int32)
    for b in range(B):
        lo, hi = int(w.node_off[b]), int(w.node_off[b + 1])
        s, depth, anc, leaf = tree(w.parent[lo:hi], shp.max_depth)
        tok = w.token[lo:hi]
        if s != 0:
            status[b] = TREE_ERROR
            continue
        if np.any(tok[1:] < 0) or np.any(tok[1:] >= shp.vocab) or np.any(w.src[lo + 1:hi] > 1):
            status[b] = TOKEN_ERROR
            continue
        if int(w.kv_len[b]) < 0 or int(w.kv_len[b]) + (hi - lo) > w.k_cache.shape[2]:
            status[b] = CAPACITY_ERROR
            continue
        f, lp, rk = node_flags(w.parent[lo:hi], tok, w.src[lo:hi], z32[lo:hi],
                               st["argmax"][lo:hi], st["lse"][lo:hi], p.topk, p.tau)
        res = path(w.parent[lo:hi], leaf, depth, f, st["argmax"][lo:hi], shp.max_depth,
                   p.min_lookahead, p.max_relaxed)
        flags[lo:hi] = f
        tok_lp[lo:hi] = lp
        tok_rank[lo:hi] = rk
        leaf_acc[lo:hi] = res["leaf_acc_len"]
        paths[b] = res["path"]
        acc_len[b] = res["acc_len"]
        bonus[b] = res["bonus"]
        winner[b] = res["winner_leaf"]
    st.update(flags=flags, tok_logprob=tok_lp, tok_rank=tok_rank, leaf_acc_len=leaf_acc,
              path=paths, acc_len=acc_len, bonus=bonus, winner_leaf=winner, seq_status=status)
    return st


def verify_step(w, params=None) -> dict:
    """Every output of one verification step for workload ``w``."""
    f = forward(w)
    d = decide(w, f["z"], params)
    d.update(attn_out=f["attn"], x=f["x"], logits=f["z"])
    return d
