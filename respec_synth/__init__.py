"""Seeded synthetic inputs for draft-tree verification.

This module is shared by the CPU oracle's tests and by the GPU path's tests
and benchmark.  It draws random numbers and builds tree shapes; it holds none
of the verification arithmetic (no attention, no logits, no softmax, no
acceptance rule).  Steps that need the target model's argmax take it as an
argument.

Random numbers come from one counter-based generator: the SplitMix64 output
sequence (Steele, Lea, Flood, "Fast splittable pseudorandom number
generators", OOPSLA 2014; Vigna's public-domain splitmix64.c).  Element ``i``
of stream ``s`` under seed ``seed`` is

    key   = mix(seed * 2**32 + s + GAMMA)
    u64_i = mix(key + (i + 1) * GAMMA)            (all arithmetic mod 2**64)

so any element can be drawn independently of the others.  Uniforms in (0, 1]
are ``((u64 >> 11) + 1) * 2**-53``; standard normals use the cosine branch of
Box-Muller on elements ``2i`` and ``2i + 1``.  Reals are rounded to float32
(round-to-nearest-even) and, for bf16 workloads, then to bf16 (RNE on the
float32 bit pattern).  bf16 tensors are returned as ``uint16`` bit patterns.

Workload shapes stand in for the paper's target models (Vicuna-7B,
Qwen2-7B, Llama-3.1-8B shapes; Section 4.1) and its Spec-Bench traffic; no
benchmark item is used.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass, field

import numpy as np

__all__ = [
    "GAMMA", "u64_stream", "uniform_stream", "normal_stream",
    "f32_to_bf16_bits", "bf16_bits_to_f32", "SRC_MODEL", "SRC_RETRIEVED",
    "Shape", "AcceptParams", "Workload", "CONFIGS", "generate",
    "apply_prefix_rule", "redraw_hidden_row", "redraw_token", "token_stream_value",
    "STREAM", "custom", "build",
]

GAMMA = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)
_S30, _S27, _S31, _S11 = (np.uint64(30), np.uint64(27), np.uint64(31), np.uint64(11))

SRC_MODEL = 0
SRC_RETRIEVED = 1

# Stream identifiers: one independent sequence per kind of random draw.
STREAM = {
    "hidden": 1, "k_cache": 2, "v_cache": 3, "lm_head": 4, "tree": 5,
    "tags": 6, "tokens": 7, "kv_len": 8, "prefix": 9, "repair_hidden": 10,
    "repair_token": 11, "zipf": 12, "exercise": 13, "accept_len": 14,
}

_CHUNK = 1 << 22

_HERE = os.path.dirname(os.path.abspath(__file__))
_SO = os.path.join(_HERE, "_synth_gen.so")
_LIB = None


def build(force: bool = False) -> str:
    """Compile the C sampling helper next to this file (gcc, OpenMP)."""
    src = os.path.join(_HERE, "synth_gen.c")
    if force or not os.path.exists(_SO) or os.path.getmtime(_SO) < os.path.getmtime(src):
        tmp = _SO + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-std=gnu11", "-O2", "-fopenmp", "-fPIC", "-shared",
                               "-ffp-contract=off", src, "-o", tmp, "-lm"])
        os.replace(tmp, _SO)
    return _SO


def _lib():
    global _LIB
    if _LIB is None:
        build()
        lib = ctypes.CDLL(_SO)
        for name, ptr_t in (("synth_normal_f32", ctypes.c_void_p), ("synth_normal_bf16", ctypes.c_void_p)):
            fn = getattr(lib, name)
            fn.argtypes = [ctypes.c_uint64, ctypes.c_uint32, ctypes.c_uint64, ctypes.c_int64,
                           ctypes.c_double, ptr_t]
            fn.restype = None
        _LIB = lib
    return _LIB


def _ptr(a: np.ndarray) -> int:
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data



def _mix(z: np.ndarray) -> np.ndarray:
    z = (z ^ (z >> _S30)) * _M1
    z = (z ^ (z >> _S27)) * _M2
    return z ^ (z >> _S31)


def _key(seed: int, stream: int) -> np.uint64:
    s = np.array([((seed & 0xFFFFFFFF) << 32) + (stream & 0xFFFFFFFF)], dtype=np.uint64)
    with np.errstate(over="ignore"):
        return _mix(s + GAMMA)[0]


def u64_stream(seed: int, stream: int, start: int, count: int) -> np.ndarray:
    """Elements ``start .. start+count-1`` of a SplitMix64 stream (uint64)."""
    key = _key(seed, stream)
    idx = np.arange(start + 1, start + 1 + count, dtype=np.uint64)
    with np.errstate(over="ignore"):
        return _mix(key + idx * GAMMA)


def uniform_stream(seed: int, stream: int, start: int, count: int) -> np.ndarray:
    """Uniform doubles in (0, 1] from the 53 high bits of each element."""
    u = u64_stream(seed, stream, start, count)
    return ((u >> _S11).astype(np.float64) + 1.0) * (2.0 ** -53)


def normal_stream(seed: int, stream: int, start: int, count: int) -> np.ndarray:
    """Standard normals (Box-Muller, cosine branch) for indices start..start+count-1.

    Computed by the C helper (float64, libm) and returned as float64 only
    after rounding to float32, the precision every workload tensor uses.
    """
    out = np.empty(count, dtype=np.float32)
    _lib().synth_normal_f32(seed, stream, start, count, 1.0, _ptr(out))
    return out.astype(np.float64)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (round-to-nearest-even); returns uint16 bits."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    b = b + np.uint64(0x7FFF) + ((b >> np.uint64(16)) & np.uint64(1))
    return (b >> np.uint64(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _real_tensor(seed, stream, shape, std, dtype):
    n = int(np.prod(shape))
    if dtype == "bf16":
        out = np.empty(n, dtype=np.uint16)
        _lib().synth_normal_bf16(seed, stream, 0, n, float(std), _ptr(out))
    else:
        out = np.empty(n, dtype=np.float32)
        _lib().synth_normal_f32(seed, stream, 0, n, float(std), _ptr(out))
    return out.reshape(shape)


# ----------------------------------------------------------------------------
# Workload description
# ----------------------------------------------------------------------------

@dataclass(frozen=True)
class Shape:
    name: str
    dtype: str            # "f32" or "bf16"
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    vocab: int
    batch: int
    max_nodes: int        # nodes per tree (capacity)
    max_depth: int
    topk_out: int = 8


@dataclass(frozen=True)
class AcceptParams:
    topk: int = 8         # k of TopK_k in the relaxed check (Section 3.4)
    tau: float = 3.0      # tolerance margin tau (Section 3.4)
    min_lookahead: int = 2  # m: greedy matches required after a relaxed token
    max_relaxed: int = 2    # Phi: number of relaxed attempts
    stochastic: int = 0     # 1: speculative-sampling verification (Section 3.4, drafter outputs)
    temperature: float = 1.0


@dataclass
class Workload:
    shape: Shape
    seed: int
    hidden: np.ndarray     # [M][Hd]   (uint16 bf16 bits or float32)
    k_cache: np.ndarray    # [B][Hkv][L_cap][D]
    v_cache: np.ndarray    # [B][Hkv][L_cap][D]
    lm_head: np.ndarray    # [V][Hd]
    parent: np.ndarray     # [M] int32, sequence-local parent index, root = -1
    node_off: np.ndarray   # [B+1] int32
    kv_len: np.ndarray     # [B] int32, prefix length L_b
    src: np.ndarray        # [M] uint8 (SRC_MODEL / SRC_RETRIEVED)
    token: np.ndarray      # [M] int32 draft token of each node (root's is the last verified token)
    params: AcceptParams = field(default_factory=AcceptParams)
    prefix_plan: dict = field(default_factory=dict)

    @property
    def kv_cap(self) -> int:
        return int(self.k_cache.shape[2])

    @property
    def total_nodes(self) -> int:
        return int(self.node_off[-1])


def _cfg_shapes():
    b7 = dict(hidden=4096, n_q_heads=32, n_kv_heads=32, head_dim=128, vocab=32000)
    return {
        0: Shape("tiny-f32", "f32", 256, 4, 4, 64, 4096, 1, 16, 5),
        1: Shape("7b-26node-L2048", "bf16", batch=1, max_nodes=26, max_depth=6, **b7),
        2: Shape("7b-65node-L16384", "bf16", batch=1, max_nodes=65, max_depth=8, **b7),
        3: Shape("7b-batch8x32-ragged", "bf16", batch=8, max_nodes=32, max_depth=7, **b7),
        4: Shape("llama3-8b-gqa-64node-L32768", "bf16", 4096, 32, 8, 128, 128256, 1, 64, 8),
    }


CONFIGS = _cfg_shapes()
SEED_BASE = 12820


# ----------------------------------------------------------------------------
# Tree shapes (sequence-local parent arrays, parent[j] < j)
# ----------------------------------------------------------------------------

def _chains(n_chains, depth, first=1):
    parent = []
    for c in range(n_chains):
        base = first + c * depth
        for d in range(depth):
            parent.append(0 if d == 0 else base + d - 1)
    return parent


def _random_tree(seed, stream_off, n_nodes, max_depth, max_branch):
    """Random parent array: node j picks a uniform earlier node with room."""
    parent = [-1]
    depth = [0] * len(parent)
    for j in range(1, len(parent)):
        depth[j] = depth[parent[j]] + 1
    nchild = [0] * len(parent)
    for j in range(1, len(parent)):
        nchild[parent[j]] += 1
    u = uniform_stream(seed, STREAM["tree"], stream_off, n_nodes)
    for j in range(len(parent), n_nodes):
        cand = [i for i in range(j) if depth[i] < max_depth and nchild[i] < max_branch]
        pick = cand[min(int(u[j] * len(cand)), len(cand) - 1)]
        parent.append(pick)
        depth.append(depth[pick] + 1)
        nchild.append(0)
        nchild[pick] += 1
    return parent


def _permutation(seed, stream, off, n):
    u = uniform_stream(seed, stream, off, n)
    p = list(range(n))
    for i in range(n - 1, 0, -1):
        j = min(int(u[i] * (i + 1)), i)
        p[i], p[j] = p[j], p[i]
    return p


def _zipf_tokens(seed, off, n, vocab, s=1.1):
    ranks = np.arange(1, vocab + 1, dtype=np.float64)
    cdf = np.cumsum(ranks ** -s)
    cdf /= cdf[-1]
    u = uniform_stream(seed, STREAM["zipf"], off, n)
    return np.minimum(np.searchsorted(cdf, u, side="left"), vocab - 1).astype(np.int32)


def generate(config: int, *, params: AcceptParams | None = None, seed: int | None = None,
             poison_tail: bool = False) -> Workload:
    """Build the seeded inputs of one workload (before any argmax-dependent step).

    ``poison_tail`` fills K/V rows beyond L_b + N_b with NaN so that a kernel
    reading past a sequence's end shows up in the results.
    """
    shp = CONFIGS[config]
    seed = SEED_BASE + config if seed is None else seed
    if params is None:
        params = AcceptParams()
    B = shp.batch
    plan = {}

    if config == 0:
        parents = [[-1] + _chains(3, 5)]
        src = [[SRC_MODEL] + [SRC_RETRIEVED] * 10 + [SRC_MODEL] * 5]
        kv = [512]
        plan = {"kind": "chains", "chains": [list(range(1 + 5 * c, 6 + 5 * c)) for c in range(3)]}
    elif config == 1:
        par = _random_tree(seed, 0, 26, 6, 4)
        perm = _permutation(seed, STREAM["tags"], 0, 25)
        tags = [SRC_MODEL] * 26
        for p in perm[:13]:
            tags[1 + p] = SRC_RETRIEVED
        parents, src, kv = [par], [tags], [2048]
        plan = {"kind": "tree"}
    elif config == 2:
        parents = [[-1] + _chains(8, 8)]
        src = [[SRC_MODEL] + [SRC_RETRIEVED] * 64]
        kv = [16384]
        alen = np.minimum((uniform_stream(seed, STREAM["accept_len"], 0, 8) * 9).astype(np.int64), 8)
        plan = {"kind": "chains_exact", "chains": [list(range(1 + 8 * c, 9 + 8 * c)) for c in range(8)],
                "accept_len": [int(a) for a in alen]}
    elif config == 3:
        parents, src = [], []
        kvu = uniform_stream(seed, STREAM["kv_len"], 0, B)
        kv = [1024 + min(int(u * 7169), 7168) for u in kvu]
        for b in range(B):
            parents.append(_random_tree(seed, 1000 * (b + 1), 32, 7, 4))
            tu = uniform_stream(seed, STREAM["tags"], 1000 * (b + 1), 32)
            src.append([SRC_MODEL] + [SRC_RETRIEVED if tu[j] < 0.5 else SRC_MODEL for j in range(1, 32)])
        plan = {"kind": "tree"}
    elif config == 4:
        base = [-1] + _chains(6, 8)
        # the model subtree counts branching among model nodes only: the
        # root's six chain children do not use up its branching budget.
        par = _model_subtree(seed, base, 64, 5, 4)
        parents = [par]
        src = [[SRC_MODEL] + [SRC_RETRIEVED] * 48 + [SRC_MODEL] * 15]
        kv = [32768]
        plan = {"kind": "mixed", "chains": [list(range(1 + 8 * c, 9 + 8 * c)) for c in range(6)]}
    else:
        raise ValueError(f"unknown config {config}")

    node_off = np.zeros(B + 1, dtype=np.int32)
    for b in range(B):
        node_off[b + 1] = node_off[b] + len(parents[b])
    M = int(node_off[-1])
    L_cap = max(kv[b] + len(parents[b]) for b in range(B))
    Hd, Hkv, D, V = shp.hidden, shp.n_kv_heads, shp.head_dim, shp.vocab

    hidden = _real_tensor(seed, STREAM["hidden"], (M, Hd), 1.0, shp.dtype)
    kc = _real_tensor(seed, STREAM["k_cache"], (B, Hkv, L_cap, D), 1.0, shp.dtype)
    vc = _real_tensor(seed, STREAM["v_cache"], (B, Hkv, L_cap, D), 1.0, shp.dtype)
    W = _real_tensor(seed, STREAM["lm_head"], (V, Hd), 0.02, shp.dtype)
    if poison_tail:
        nan = np.uint16(0x7FC0) if shp.dtype == "bf16" else np.float32(np.nan)
        for b in range(B):
            end = kv[b] + len(parents[b])
            kc[b, :, end:, :] = nan
            vc[b, :, end:, :] = nan

    parent = np.concatenate([np.asarray(p, dtype=np.int32) for p in parents])
    srcs = np.concatenate([np.asarray(s, dtype=np.uint8) for s in src])
    if config == 2:
        token = _zipf_tokens(seed, 0, M, V)
    else:
        token = np.minimum((uniform_stream(seed, STREAM["tokens"], 0, M) * V).astype(np.int64), V - 1).astype(np.int32)

    return Workload(shp, seed, hidden, kc, vc, W, parent, node_off,
                    np.asarray(kv, dtype=np.int32), srcs, token, params, plan)


def _model_subtree(seed, base, n_nodes, max_depth, max_branch):
    parent = list(base)
    depth = [0] * len(parent)
    for j in range(1, len(parent)):
        depth[j] = depth[parent[j]] + 1
    model_nodes = [0]
    nchild = {0: 0}
    u = uniform_stream(seed, STREAM["tree"], 0, n_nodes)
    for j in range(len(base), n_nodes):
        cand = [i for i in model_nodes if depth[i] < max_depth and nchild[i] < max_branch]
        pick = cand[min(int(u[j] * len(cand)), len(cand) - 1)]
        parent.append(pick)
        depth.append(depth[pick] + 1)
        nchild[pick] += 1
        nchild[j] = 0
        model_nodes.append(j)
    return parent


# ----------------------------------------------------------------------------
# Argmax-dependent token assignment and repair draws
# ----------------------------------------------------------------------------

def token_stream_value(w: Workload, stream: str, index: int, vocab: int | None = None) -> int:
    V = w.shape.vocab if vocab is None else vocab
    u = uniform_stream(w.seed, STREAM[stream], index, 1)[0]
    return min(int(u * V), V - 1)


def apply_prefix_rule(w: Workload, argmax: np.ndarray) -> np.ndarray:
    """Replace seeded draft prefixes by the target's argmax at the parent.

    ``argmax[i]`` is the target's greedy next token after node ``i`` (global
    node index).  Chains: each chain is picked with probability 1/2 and a
    prefix of uniform length 1..depth is replaced.  Trees: a child of the
    root, or of a replaced node, is replaced with probability 1/2.  For
    exact-length chains the first A tokens are replaced and token A+1 is made
    to differ from the argmax.  Returns the new token array.
    """
    tok = w.token.copy()
    plan = w.prefix_plan
    kind = plan.get("kind", "tree")
    u = uniform_stream(w.seed, STREAM["prefix"], 0, max(4 * w.total_nodes, 64))
    if kind in ("chains", "mixed"):
        chains = plan["chains"]
        for c, nodes in enumerate(chains):
            if u[2 * c] < 0.5:
                plen = 1 + min(int(u[2 * c + 1] * len(nodes)), len(nodes) - 1)
                for n in nodes[:plen]:
                    tok[n] = argmax[w.parent[n]]
        if kind == "mixed":
            chain_nodes = {n for ch in chains for n in ch}
            _tree_rule(w, tok, argmax, u, 2 * len(chains), skip=chain_nodes)
    elif kind == "chains_exact":
        for c, nodes in enumerate(plan["chains"]):
            a = plan["accept_len"][c]
            for n in nodes[:a]:
                tok[n] = argmax[w.parent[n]]
            if a < len(nodes):
                n = nodes[a]
                attempt = 0
                while tok[n] == argmax[w.parent[n]]:
                    tok[n] = token_stream_value(w, "repair_token", n * 64 + attempt)
                    attempt += 1
    else:
        _tree_rule(w, tok, argmax, u, 0, skip=set())
    return tok


def _tree_rule(w, tok, argmax, u, uoff, skip):
    for b in range(len(w.node_off) - 1):
        lo, hi = int(w.node_off[b]), int(w.node_off[b + 1])
        replaced = {lo}
        for j in range(lo + 1, hi):
            if j in skip:
                continue
            p = lo + int(w.parent[j])
            if p in replaced and u[uoff + j] < 0.5:
                tok[j] = argmax[p]
                replaced.add(j)


def redraw_hidden_row(w: Workload, row: int, attempt: int) -> np.ndarray:
    """A fresh hidden-state row (same distribution) from the repair stream."""
    Hd = w.shape.hidden
    start = (row * 16 + attempt) * Hd
    vals = normal_stream(w.seed, STREAM["repair_hidden"], start, Hd).astype(np.float32)
    return f32_to_bf16_bits(vals) if w.shape.dtype == "bf16" else vals


def redraw_token(w: Workload, node: int, attempt: int) -> int:
    return token_stream_value(w, "repair_token", node * 64 + attempt + 32)


def custom(shape: Shape, parents, kv_len, src=None, *, seed: int = 7, params: AcceptParams | None = None,
           poison_tail: bool = False, tokens=None) -> Workload:
    """A workload with caller-chosen shapes and trees (edge cases, pins).

    ``parents`` is a list of per-sequence parent arrays, ``kv_len`` the
    prefix length of each sequence, ``src`` optional per-sequence tag lists
    (default: all retrieved except the root).  Tensors are drawn exactly as in
    ``generate`` (N(0,1) hidden/K/V, N(0, 0.02^2) LM head).
    """
    B = len(parents)
    node_off = np.zeros(B + 1, dtype=np.int32)
    for b in range(B):
        node_off[b + 1] = node_off[b] + len(parents[b])
    M = int(node_off[-1])
    L_cap = max([kv_len[b] + len(parents[b]) for b in range(B)] + [1])
    Hd, Hkv, D, V = shape.hidden, shape.n_kv_heads, shape.head_dim, shape.vocab
    hidden = _real_tensor(seed, STREAM["hidden"], (M, Hd), 1.0, shape.dtype)
    kc = _real_tensor(seed, STREAM["k_cache"], (B, Hkv, L_cap, D), 1.0, shape.dtype)
    vc = _real_tensor(seed, STREAM["v_cache"], (B, Hkv, L_cap, D), 1.0, shape.dtype)
    W = _real_tensor(seed, STREAM["lm_head"], (V, Hd), 0.02, shape.dtype)
    if poison_tail:
        nan = np.uint16(0x7FC0) if shape.dtype == "bf16" else np.float32(np.nan)
        for b in range(B):
            end = kv_len[b] + len(parents[b])
            kc[b, :, end:, :] = nan
            vc[b, :, end:, :] = nan
    parent = np.concatenate([np.asarray(p, dtype=np.int32) for p in parents]) if M else np.zeros(0, np.int32)
    if src is None:
        src = [[SRC_MODEL] + [SRC_RETRIEVED] * (len(p) - 1) for p in parents]
    srcs = np.concatenate([np.asarray(s, dtype=np.uint8) for s in src]) if M else np.zeros(0, np.uint8)
    if tokens is None:
        token = np.minimum((uniform_stream(seed, STREAM["tokens"], 0, max(M, 1)) * V).astype(np.int64),
                           V - 1).astype(np.int32)[:M]
    else:
        token = np.asarray(tokens, dtype=np.int32)
    return Workload(shape, seed, hidden, kc, vc, W, parent, node_off,
                    np.asarray(kv_len, dtype=np.int32), srcs, token,
                    AcceptParams() if params is None else params, {"kind": "tree"})
