"""ctypes binding of the drafting side of librespec_verify.so (include/respec_draft.h).

Argument marshalling only: the trigger (Eq. 1-3), the suffix automaton, the
EMA scores and selection (Eq. 4-5), BuildDraftTree and the per-sequence
session all run in the library's C++ code.  Every array is host memory.
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass, field

import numpy as np

from .binding import OK, lib as _verify_lib, VerifyError

MAX_SELECT = 16
_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64


class TriggerParams(ctypes.Structure):
    _fields_ = [("max_lookback", _I32), ("lambda_e", ctypes.c_float), ("theta_entropy", ctypes.c_float)]


class TriggerResult(ctypes.Structure):
    _fields_ = [("key_len", _I32), ("h_min", ctypes.c_float), ("c_min", ctypes.c_float), ("fire", _I32)]


class SelectParams(ctypes.Structure):
    _fields_ = [("alpha", ctypes.c_float), ("theta_score", ctypes.c_float), ("s0", ctypes.c_float),
                ("n_select", _I32)]


class TreeParams(ctypes.Structure):
    _fields_ = [("max_draft_len", _I32), ("max_nodes", _I32)]


class DraftParams(ctypes.Structure):
    _fields_ = [("trigger", TriggerParams), ("select", SelectParams), ("tree", TreeParams)]


class DraftResult(ctypes.Structure):
    _fields_ = [("retrieved", _I32), ("trigger", TriggerResult), ("n_positions", _I32), ("n_selected", _I32),
                ("sel_pos", _I32 * MAX_SELECT), ("cand_end", _I32 * MAX_SELECT), ("cand_len", _I32 * MAX_SELECT),
                ("n_nodes", _I32)]


_READY = False


def lib() -> ctypes.CDLL:
    global _READY
    L = _verify_lib()
    if not _READY:
        sig = {
            "respec_trigger_eval": (ctypes.c_int, [_P, _I32, ctypes.POINTER(TriggerParams),
                                                   ctypes.POINTER(TriggerResult)]),
            "respec_sam_create": (ctypes.c_int, [ctypes.POINTER(_P)]),
            "respec_sam_destroy": (None, [_P]),
            "respec_sam_extend": (ctypes.c_int, [_P, _P, _I32]),
            "respec_sam_length": (_I64, [_P]),
            "respec_sam_text": (ctypes.c_int, [_P, _I64, _I32, _P]),
            "respec_sam_positions": (ctypes.c_int, [_P, _P, _I32, _P, _I32, ctypes.POINTER(_I32)]),
            "respec_scores_create": (ctypes.c_int, [ctypes.POINTER(_P)]),
            "respec_scores_destroy": (None, [_P]),
            "respec_scores_get": (ctypes.c_double, [_P, _I32, ctypes.c_double]),
            "respec_scores_size": (_I64, [_P]),
            "respec_select": (ctypes.c_int, [_P, _P, _I32, ctypes.POINTER(SelectParams), _P, ctypes.POINTER(_I32)]),
            "respec_scores_update": (ctypes.c_int, [_P, _P, _I32, _I32, _I32, _P, ctypes.POINTER(SelectParams)]),
            "respec_build_tree": (ctypes.c_int, [_P, _P, _I32, ctypes.POINTER(TreeParams), _P, _P, _P,
                                                 ctypes.POINTER(_I32), _P, _P]),
            "respec_draft_session_create": (ctypes.c_int, [ctypes.POINTER(DraftParams), ctypes.POINTER(_P)]),
            "respec_draft_session_destroy": (None, [_P]),
            "respec_draft_session_append": (ctypes.c_int, [_P, _P, _P, _I32]),
            "respec_draft_session_propose": (ctypes.c_int, [_P, _P, _P, _P, _I32, ctypes.POINTER(DraftResult)]),
            "respec_draft_session_commit": (ctypes.c_int, [_P, _P, _P, _I32, _I32, _P]),
            "respec_draft_session_sam": (_P, [_P]),
            "respec_draft_session_scores": (_P, [_P]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _READY = True
    return L


DRAFT_EXPORTS = (
    "respec_trigger_eval", "respec_sam_create", "respec_sam_destroy", "respec_sam_extend", "respec_sam_length",
    "respec_sam_text", "respec_sam_positions", "respec_scores_create", "respec_scores_destroy",
    "respec_scores_get", "respec_scores_size", "respec_select", "respec_scores_update", "respec_build_tree",
    "respec_draft_session_create", "respec_draft_session_destroy", "respec_draft_session_append",
    "respec_draft_session_propose", "respec_draft_session_commit", "respec_draft_session_sam",
    "respec_draft_session_scores",
)


def _check(status: int, where: str) -> None:
    if status != OK:
        raise VerifyError(status, where)


def _i32(a):
    return np.ascontiguousarray(a, dtype=np.int32)


def _ptr(a):
    return a.ctypes.data if a.size else None


@dataclass
class Trigger:
    key_len: int
    h_min: float
    c_min: float
    fire: bool


def trigger_eval(entropy, max_lookback=3, lambda_e=0.5, theta_entropy=1.5) -> Trigger:
    """Entropy-guided trigger (Eq. 1-3) over the entropies of the context's last tokens."""
    e = np.ascontiguousarray(entropy, dtype=np.float32)
    r = TriggerResult()
    p = TriggerParams(max_lookback, lambda_e, theta_entropy)
    _check(lib().respec_trigger_eval(_ptr(e), int(e.size), ctypes.byref(p), ctypes.byref(r)), "respec_trigger_eval")
    return Trigger(int(r.key_len), float(r.h_min), float(r.c_min), bool(r.fire))


class Sam:
    """Suffix automaton of a token context (owned, or a session's view)."""

    def __init__(self, tokens=None, *, _view=None):
        self._own = _view is None
        if _view is None:
            h = _P()
            _check(lib().respec_sam_create(ctypes.byref(h)), "respec_sam_create")
            self._h = h
        else:
            self._h = _P(_view)
        if tokens is not None:
            self.extend(tokens)

    def __del__(self):
        try:
            if getattr(self, "_own", False) and getattr(self, "_h", None):
                lib().respec_sam_destroy(self._h)
                self._h = None
        except Exception:   # interpreter shutdown
            pass

    def extend(self, tokens) -> None:
        t = _i32(tokens)
        _check(lib().respec_sam_extend(self._h, _ptr(t), int(t.size)), "respec_sam_extend")

    def __len__(self) -> int:
        return int(lib().respec_sam_length(self._h))

    def text(self, start=0, n=None) -> np.ndarray:
        n = len(self) - start if n is None else n
        out = np.empty(max(n, 0), np.int32)
        _check(lib().respec_sam_text(self._h, int(start), int(n), _ptr(out)), "respec_sam_text")
        return out

    def positions(self, key, cap=None) -> np.ndarray:
        """Retrieval positions of key, most recent first (all of them unless cap is given)."""
        k = _i32(key)
        total = _I32()
        _check(lib().respec_sam_positions(self._h, _ptr(k), int(k.size), None, 0, ctypes.byref(total)),
               "respec_sam_positions")
        m = int(total.value) if cap is None else min(int(cap), int(total.value))
        out = np.empty(m, np.int32)
        _check(lib().respec_sam_positions(self._h, _ptr(k), int(k.size), _ptr(out), m, ctypes.byref(total)),
               "respec_sam_positions")
        return out


class Scores:
    """EMA score table S_pos (owned, or a session's view)."""

    def __init__(self, *, _view=None):
        self._own = _view is None
        if _view is None:
            h = _P()
            _check(lib().respec_scores_create(ctypes.byref(h)), "respec_scores_create")
            self._h = h
        else:
            self._h = _P(_view)

    def __del__(self):
        try:
            if getattr(self, "_own", False) and getattr(self, "_h", None):
                lib().respec_scores_destroy(self._h)
                self._h = None
        except Exception:   # interpreter shutdown
            pass

    def get(self, pos: int, s0: float = 0.5) -> float:
        return float(lib().respec_scores_get(self._h, int(pos), float(s0)))

    def __len__(self) -> int:
        return int(lib().respec_scores_size(self._h))

    def select(self, positions, alpha=0.5, theta_score=0.1, s0=0.5, n_select=3) -> np.ndarray:
        pos = _i32(positions)
        out = np.empty(MAX_SELECT, np.int32)
        n = _I32()
        p = SelectParams(alpha, theta_score, s0, n_select)
        _check(lib().respec_select(self._h, _ptr(pos), int(pos.size), ctypes.byref(p), out.ctypes.data,
                                   ctypes.byref(n)), "respec_select")
        return out[:n.value].copy()

    def update(self, selected, winner, l_acc, l_draft, alpha=0.5, theta_score=0.1, s0=0.5, n_select=3) -> None:
        sel = _i32(selected)
        ld = _i32(l_draft) if l_draft is not None else np.zeros(0, np.int32)
        p = SelectParams(alpha, theta_score, s0, n_select)
        _check(lib().respec_scores_update(self._h, _ptr(sel), int(sel.size), int(winner), int(l_acc), _ptr(ld),
                                          ctypes.byref(p)), "respec_scores_update")


@dataclass
class DraftTree:
    parent: np.ndarray
    token: np.ndarray
    src: np.ndarray
    cand_end: np.ndarray = field(default_factory=lambda: np.zeros(0, np.int32))
    cand_len: np.ndarray = field(default_factory=lambda: np.zeros(0, np.int32))


def build_tree(sam: Sam, selected, max_draft_len=20, max_nodes=61) -> DraftTree:
    """BuildDraftTree: trie merge of the selected continuations, rooted at the last token."""
    sel = _i32(selected)
    parent = np.empty(max_nodes, np.int32)
    token = np.empty(max_nodes, np.int32)
    src = np.empty(max_nodes, np.uint8)
    ce = np.empty(max(sel.size, 1), np.int32)
    cl = np.empty(max(sel.size, 1), np.int32)
    n = _I32()
    p = TreeParams(max_draft_len, max_nodes)
    _check(lib().respec_build_tree(sam._h, _ptr(sel), int(sel.size), ctypes.byref(p), parent.ctypes.data,
                                   token.ctypes.data, src.ctypes.data, ctypes.byref(n), ce.ctypes.data,
                                   cl.ctypes.data), "respec_build_tree")
    m = int(n.value)
    return DraftTree(parent[:m].copy(), token[:m].copy(), src[:m].copy(), ce[:sel.size].copy(), cl[:sel.size].copy())


@dataclass
class Proposal:
    retrieved: bool
    trigger: Trigger
    n_positions: int
    selected: np.ndarray
    tree: DraftTree


class DraftSession:
    """Algorithm 1's host side for one sequence (trigger, retrieval, selection, tree, feedback)."""

    def __init__(self, *, max_lookback=3, lambda_e=0.5, theta_entropy=1.5, alpha=0.5, theta_score=0.1, s0=0.5,
                 n_select=3, max_draft_len=20, max_nodes=61):
        self.params = DraftParams(TriggerParams(max_lookback, lambda_e, theta_entropy),
                                  SelectParams(alpha, theta_score, s0, n_select), TreeParams(max_draft_len, max_nodes))
        h = _P()
        _check(lib().respec_draft_session_create(ctypes.byref(self.params), ctypes.byref(h)),
               "respec_draft_session_create")
        self._h = h
        self.sam = Sam(_view=lib().respec_draft_session_sam(h))
        self.scores = Scores(_view=lib().respec_draft_session_scores(h))

    def __del__(self):
        try:
            if getattr(self, "_h", None):
                lib().respec_draft_session_destroy(self._h)
                self._h = None
        except Exception:   # interpreter shutdown
            pass

    def append(self, tokens, entropy=None) -> None:
        t = _i32(tokens)
        e = None if entropy is None else np.ascontiguousarray(entropy, dtype=np.float32)
        _check(lib().respec_draft_session_append(self._h, _ptr(t), None if e is None else _ptr(e), int(t.size)),
               "respec_draft_session_append")

    def propose(self) -> Proposal:
        cap = self.params.tree.max_nodes
        parent = np.empty(cap, np.int32)
        token = np.empty(cap, np.int32)
        src = np.empty(cap, np.uint8)
        r = DraftResult()
        _check(lib().respec_draft_session_propose(self._h, parent.ctypes.data, token.ctypes.data, src.ctypes.data,
                                                  cap, ctypes.byref(r)), "respec_draft_session_propose")
        m, ns = int(r.n_nodes), int(r.n_selected)
        tr = Trigger(int(r.trigger.key_len), float(r.trigger.h_min), float(r.trigger.c_min), bool(r.trigger.fire))
        tree = DraftTree(parent[:m].copy(), token[:m].copy(), src[:m].copy(),
                         np.array(r.cand_end[:ns], np.int32), np.array(r.cand_len[:ns], np.int32))
        return Proposal(bool(r.retrieved), tr, int(r.n_positions), np.array(r.sel_pos[:ns], np.int32), tree)

    def commit(self, token, path, acc_len: int, bonus: int, entropy) -> None:
        t = _i32(token)
        pa = _i32(path)
        e = np.ascontiguousarray(entropy, dtype=np.float32)
        _check(lib().respec_draft_session_commit(self._h, _ptr(t), _ptr(pa), int(acc_len), int(bonus), _ptr(e)),
               "respec_draft_session_commit")
