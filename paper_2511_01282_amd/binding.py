"""ctypes binding of librespec_verify.so (argument marshalling only).

Every computation of the verification step runs in the library's HIP kernels;
this module only builds the C structs of ``include/respec_verify.h`` from
torch tensors (device memory and streams) and raises on non-OK statuses.
Importing it fails loudly when the library has not been built.
"""
from __future__ import annotations

import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "librespec_verify.so")

(OK, ERR_NULL, ERR_SHAPE, ERR_DTYPE, ERR_PARAM, ERR_TREE, ERR_CAPACITY, ERR_HIP, ERR_WORKSPACE, ERR_TOKEN,
 ERR_SCRATCH) = range(11)
NOALLOC_SCRATCH_BYTES, NOALLOC_MAX_BATCH = 64 << 20, 16384
F32, BF16 = 0, 1
SRC_MODEL, SRC_RETRIEVED = 0, 1
FLAG_GREEDY, FLAG_TOPK, FLAG_TAU, FLAG_RELAXED, FLAG_ON_PATH, FLAG_STOCH_ACCEPT = 1, 2, 4, 8, 16, 32
STOP_ALL, STOP_ATTN, STOP_LOGITS, STOP_STATS = 0, 1, 2, 3
MAX_NODES, MAX_DEPTH, MAX_TOPK_OUT = 128, 64, 16

EXPORTS = (
    "respec_verify_create", "respec_verify_destroy", "respec_verify_workspace_bytes",
    "respec_verify_workspace_init", "respec_verify_check_tree", "respec_verify_step",
    "respec_verify_step_noalloc", "respec_status_string",
)


class Shape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "hidden", "n_q_heads", "n_kv_heads", "head_dim", "vocab", "dtype", "max_batch",
        "max_nodes", "max_depth", "max_kv_len", "topk_out")]


class AcceptParams(ctypes.Structure):
    _fields_ = [("topk", ctypes.c_int32), ("tau", ctypes.c_float),
                ("min_lookahead", ctypes.c_int32), ("max_relaxed", ctypes.c_int32),
                ("stochastic", ctypes.c_int32), ("temperature", ctypes.c_float)]


_P = ctypes.c_void_p


class Args(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32), ("total_nodes", ctypes.c_int32),
        ("max_nodes_in_batch", ctypes.c_int32), ("max_kv_len_in_batch", ctypes.c_int32),
        ("kv_capacity", ctypes.c_int32), ("stop_after", ctypes.c_int32),
        ("accept", AcceptParams),
        ("node_off", _P), ("kv_len", _P), ("hidden", _P), ("k_cache", _P), ("v_cache", _P),
        ("lm_head", _P), ("parent", _P), ("token", _P), ("src", _P), ("draft_prob", _P), ("uniform", _P),
        ("attn_out", _P), ("x_out", _P), ("logits", _P), ("max_logit", _P), ("lse", _P), ("entropy", _P),
        ("argmax", _P), ("topk_id", _P), ("topk_logprob", _P), ("tok_logprob", _P), ("tok_rank", _P),
        ("flags", _P),
        ("leaf_acc_len", _P), ("path", _P), ("acc_len", _P), ("bonus", _P), ("winner_leaf", _P),
        ("seq_status", _P), ("sample", _P), ("stage_events", _P),
    ]


INPUT_FIELDS = ("node_off", "kv_len", "hidden", "k_cache", "v_cache", "lm_head", "parent", "token", "src",
                "draft_prob", "uniform")
OUTPUT_FIELDS = ("attn_out", "x_out", "logits", "max_logit", "lse", "entropy", "argmax", "topk_id",
                 "topk_logprob", "tok_logprob", "tok_rank", "flags", "leaf_acc_len", "path", "acc_len", "bonus",
                 "winner_leaf", "seq_status", "sample")

_LIB = None


def lib() -> ctypes.CDLL:
    """Load the HIP library; raises if it has not been built."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with paper_2511_01282_amd/build.py "
                              "(or __graft_entry__.build()); there is no fallback path")
        L = ctypes.CDLL(LIB_PATH)
        L.respec_verify_create.argtypes = [ctypes.POINTER(Shape), ctypes.POINTER(ctypes.c_void_p)]
        L.respec_verify_create.restype = ctypes.c_int
        L.respec_verify_destroy.argtypes = [ctypes.c_void_p]
        L.respec_verify_destroy.restype = None
        L.respec_verify_workspace_bytes.argtypes = [ctypes.c_void_p]
        L.respec_verify_workspace_bytes.restype = ctypes.c_size_t
        L.respec_verify_workspace_init.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        L.respec_verify_workspace_init.restype = ctypes.c_int
        L.respec_verify_check_tree.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32]
        L.respec_verify_check_tree.restype = ctypes.c_int
        L.respec_verify_step.argtypes = [ctypes.c_void_p, ctypes.POINTER(Args), ctypes.c_void_p, ctypes.c_void_p]
        L.respec_verify_step.restype = ctypes.c_int
        L.respec_verify_step_noalloc.argtypes = [ctypes.c_void_p, ctypes.POINTER(Args), ctypes.c_void_p]
        L.respec_verify_step_noalloc.restype = ctypes.c_int
        L.respec_status_string.argtypes = [ctypes.c_int]
        L.respec_status_string.restype = ctypes.c_char_p
        _LIB = L
    return _LIB


class VerifyError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {lib().respec_status_string(status).decode()} (status {status})")


def _check(status: int, where: str) -> None:
    if status != OK:
        raise VerifyError(status, where)


def status_string(status: int) -> str:
    return lib().respec_status_string(status).decode()


def check_tree(parent, max_depth: int) -> int:
    """Host check of one parent array (returns the status code)."""
    import numpy as np
    arr = np.ascontiguousarray(parent, dtype=np.int32)
    n = int(arr.size)
    buf = arr if n else np.zeros(1, np.int32)
    return lib().respec_verify_check_tree(buf.ctypes.data, n, int(max_depth))


def _ptr(t) -> int | None:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not t.is_cuda:
        raise ValueError("every tensor passed to the verification step must live on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensors must be contiguous")
    return t.data_ptr()


class Plan:
    """A respec_verify plan plus its device workspace."""

    def __init__(self, *, hidden, n_q_heads, n_kv_heads, head_dim, vocab, dtype, max_batch, max_nodes,
                 max_depth, max_kv_len, topk_out=8, device="cuda", workspace=None):
        self.shape = Shape(hidden, n_q_heads, n_kv_heads, head_dim, vocab, dtype, max_batch, max_nodes,
                           max_depth, max_kv_len, topk_out)
        h = ctypes.c_void_p()
        _check(lib().respec_verify_create(ctypes.byref(self.shape), ctypes.byref(h)), "respec_verify_create")
        self._h = h
        self.workspace_bytes = int(lib().respec_verify_workspace_bytes(h))
        self.device = torch.device(device)
        if workspace is None:
            buf = torch.empty(self.workspace_bytes + 256, dtype=torch.uint8, device=self.device)
            off = (-buf.data_ptr()) % 256
            self._ws_buf = buf
            self.workspace_ptr = buf.data_ptr() + off
        else:
            self._ws_buf = workspace
            self.workspace_ptr = workspace.data_ptr()
        _check(lib().respec_verify_workspace_init(h, self.workspace_ptr, self._stream(None)),
               "respec_verify_workspace_init")

    def _stream(self, stream) -> int:
        if stream is None:
            stream = torch.cuda.current_stream(self.device)
        return stream.cuda_stream

    def close(self):
        if getattr(self, "_h", None):
            lib().respec_verify_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def step(self, inputs: dict, outputs: dict, *, batch, total_nodes, max_nodes_in_batch,
             max_kv_len_in_batch, kv_capacity, topk=8, tau=3.0, min_lookahead=2, max_relaxed=2,
             stochastic=0, temperature=1.0, stop_after=STOP_ALL, stream=None, stage_events=None,
             noalloc=False) -> None:
        """Enqueue one verification step (asynchronous, on ``stream``).

        ``noalloc``: call respec_verify_step_noalloc (the library's static scratch
        instead of this plan's workspace)."""
        a = Args()
        a.batch, a.total_nodes = batch, total_nodes
        a.max_nodes_in_batch, a.max_kv_len_in_batch = max_nodes_in_batch, max_kv_len_in_batch
        a.kv_capacity, a.stop_after = kv_capacity, stop_after
        a.accept = AcceptParams(topk, tau, min_lookahead, max_relaxed, int(stochastic), temperature)
        for f in INPUT_FIELDS:
            setattr(a, f, _ptr(inputs.get(f)))
        for f in OUTPUT_FIELDS:
            setattr(a, f, _ptr(outputs.get(f)))
        ev_arr = None
        if stage_events is not None:
            ev_arr = (ctypes.c_void_p * 4)(*[e.cuda_event for e in stage_events])
            a.stage_events = ctypes.cast(ev_arr, ctypes.c_void_p)
        if noalloc:
            _check(lib().respec_verify_step_noalloc(self._h, ctypes.byref(a), self._stream(stream)),
                   "respec_verify_step_noalloc")
        else:
            _check(lib().respec_verify_step(self._h, ctypes.byref(a), self.workspace_ptr, self._stream(stream)),
                   "respec_verify_step")


def alloc_outputs(*, total_nodes, batch, hidden, vocab, topk_out, max_depth, device="cuda",
                  attn_out=True, x_dtype=None, tok_rank=False) -> dict:
    """Output tensors of one step.  ``x_dtype`` (torch.bfloat16 / torch.float32): also
    return the residual x; ``tok_rank``: also the exact ranks of the draft tokens."""
    M, B = total_nodes, batch
    f32 = dict(dtype=torch.float32, device=device)
    i32 = dict(dtype=torch.int32, device=device)
    return {
        "attn_out": torch.empty(M, hidden, **f32) if attn_out else None,
        "x_out": torch.empty(M, hidden, dtype=x_dtype, device=device) if x_dtype is not None else None,
        "tok_rank": torch.empty(M, **i32) if tok_rank else None,
        "logits": torch.empty(M, vocab, **f32),
        "max_logit": torch.empty(M, **f32), "lse": torch.empty(M, **f32), "entropy": torch.empty(M, **f32),
        "argmax": torch.empty(M, **i32),
        "topk_id": torch.empty(M, topk_out, **i32), "topk_logprob": torch.empty(M, topk_out, **f32),
        "tok_logprob": torch.empty(M, **f32), "flags": torch.empty(M, dtype=torch.uint8, device=device),
        "leaf_acc_len": torch.empty(M, **i32), "path": torch.empty(B, max_depth + 1, **i32),
        "acc_len": torch.empty(B, **i32), "bonus": torch.empty(B, **i32),
        "winner_leaf": torch.empty(B, **i32), "seq_status": torch.empty(B, **i32),
        "sample": torch.empty(M, **i32),
    }
