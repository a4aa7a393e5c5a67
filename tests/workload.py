"""Parity workloads: seeded inputs plus the oracle-driven steps that need logits.

The generator (``respec_synth``) draws every random number; this module, which
belongs to the test suite, runs the CPU oracle to

  1. keep every row's top-1 / top-2 logit gap >= MARGIN (redrawing that
     node's hidden state from the repair stream otherwise),
  2. apply the workload's argmax-prefix rule to the draft tokens,
  3. optionally steer some retrieved tokens into ranks 1..2k-1 of their
     parent's distribution followed by greedy continuations (so that the
     relaxed check and the look-ahead rule are exercised), and
  4. keep every non-greedy token's acceptance decisions >= MARGIN away from
     their thresholds: |z_top1 - z_t - tau|, and the rank-k boundary.

Logits do not depend on the draft tokens in this one-layer proxy, so tokens
can be assigned after the logits are known.  Decisions use the float32
logits, as both the oracle and the kernels do.
"""
from __future__ import annotations

import dataclasses

import numpy as np

import oracle
import respec_synth as synth

MARGIN = 1e-3


def _row_gap_ok(row32: np.ndarray) -> bool:
    top2 = np.partition(row32, -2)[-2:]
    return float(top2[1]) - float(top2[0]) >= MARGIN


def _token_ok(row32: np.ndarray, order: np.ndarray, t: int, amax: int, k: int, tau: float) -> bool:
    if t == amax:
        return True
    zt, za = float(row32[t]), float(row32[amax])
    if abs((za - zt) - tau) < MARGIN:
        return False
    r = int(np.nonzero(order == t)[0][0])
    V = row32.shape[0]
    if r < k:
        return k >= V or zt - float(row32[order[k]]) >= MARGIN
    return float(row32[order[k - 1]]) - zt >= MARGIN


def min_decision_margin(w, z) -> float:
    """Smallest distance of any decision of step ``w`` (oracle logits ``z``) from its threshold:
    every row's top-1 / top-2 gap (argmax, the bonus token) and, for every non-greedy draft
    token, its distance from the tau boundary and from the rank-k boundary."""
    p = w.params
    z32 = np.asarray(z, np.float32)
    m = np.inf
    for b in range(len(w.node_off) - 1):
        lo, hi = int(w.node_off[b]), int(w.node_off[b + 1])
        for i in range(lo, hi):
            top2 = np.partition(z32[i], -2)[-2:]
            m = min(m, float(top2[1]) - float(top2[0]))
        for j in range(lo + 1, hi):
            i = lo + int(w.parent[j])
            row, t = z32[i], int(w.token[j])
            order = _order(row)
            a = int(order[0])
            if t == a:
                continue
            zt, za = float(row[t]), float(row[a])
            m = min(m, abs((za - zt) - p.tau))
            r = int(np.nonzero(order == t)[0][0])
            if p.topk < row.shape[0]:
                m = min(m, zt - float(row[order[p.topk]]) if r < p.topk else float(row[order[p.topk - 1]]) - zt)
    return m


def _order(row32: np.ndarray) -> np.ndarray:
    ids = np.arange(row32.shape[0])
    return np.lexsort((ids, -row32.astype(np.float64)))


@dataclasses.dataclass
class Case:
    w: synth.Workload
    z: np.ndarray          # oracle float64 logits [M][V]
    attn: np.ndarray       # oracle attention output [M][Hd]
    x: np.ndarray          # oracle residual (rounded) [M][Hd]
    expected: dict         # oracle.decide(...) outputs


def build(config: int, *, params: synth.AcceptParams | None = None, exercise: bool = True,
          poison_tail: bool = True, seed: int | None = None, shape_override=None,
          tree_override=None) -> Case:
    w = synth.generate(config, params=params, seed=seed, poison_tail=poison_tail)
    if shape_override is not None:
        w = shape_override(w)
    if tree_override is not None:
        w = tree_override(w)
    return finish(w, exercise=exercise)


def finish(w: synth.Workload, *, exercise: bool = True) -> Case:
    fw = oracle.forward(w)
    z, attn, x = fw["z"], fw["attn"], fw["x"]
    M = z.shape[0]
    B = len(w.node_off) - 1
    # 1. row margins
    for attempt in range(16):
        bad = [i for i in range(M) if not _row_gap_ok(z[i].astype(np.float32))]
        if not bad:
            break
        for i in bad:
            w.hidden[i] = synth.redraw_hidden_row(w, i, attempt)
        rows_per_seq = []
        for b in range(B):
            lo, hi = int(w.node_off[b]), int(w.node_off[b + 1])
            rows_per_seq.append(np.array([i - lo for i in bad if lo <= i < hi], dtype=np.int32))
        for b in range(B):
            if rows_per_seq[b].size == 0:
                rows_per_seq[b] = np.zeros(0, np.int32)
        part = _forward_rows(w, rows_per_seq)
        for i, (a, xx, zz) in part.items():
            attn[i], x[i], z[i] = a, xx, zz
    else:
        raise RuntimeError("row margin repair did not converge")
    z32 = z.astype(np.float32)
    amax = np.array([int(np.argmax(z32[i])) for i in range(M)], dtype=np.int32)
    # 2. argmax-prefix rule
    w.token = synth.apply_prefix_rule(w, amax)
    # 3. relaxed exercise
    p = w.params
    if exercise:
        _exercise(w, z32, amax)
    # 4. token margins
    for b in range(B):
        lo, hi = int(w.node_off[b]), int(w.node_off[b + 1])
        for j in range(lo + 1, hi):
            i = lo + int(w.parent[j])
            row = z32[i]
            order = _order(row)
            attempt = 0
            while not _token_ok(row, order, int(w.token[j]), int(amax[i]), p.topk, p.tau):
                t = synth.redraw_token(w, j, attempt)
                attempt += 1
                if t != amax[i]:
                    w.token[j] = t
                if attempt > 60:
                    raise RuntimeError("token margin repair did not converge")
    exp = oracle.decide(w, z)
    return Case(w, z, attn, x, exp)


def _forward_rows(w, rows_per_seq):
    res = {}
    shp = w.shape
    dt = oracle.BF16 if shp.dtype == "bf16" else oracle.F32
    for b, rows in enumerate(rows_per_seq):
        if rows.size == 0:
            continue
        lo, hi = int(w.node_off[b]), int(w.node_off[b + 1])
        st, depth, anc, leaf = oracle.tree(w.parent[lo:hi], shp.max_depth)
        if st != 0:
            anc = np.eye(hi - lo, dtype=np.uint8)
        o = oracle.attention(dt, w.hidden[lo:hi], w.k_cache[b], w.v_cache[b], int(w.kv_len[b]),
                             anc, shp.n_q_heads, shp.n_kv_heads, shp.head_dim, rows)
        x = oracle.residual(dt, w.hidden[lo:hi][rows], o)
        z = oracle.logits(dt, x, w.lm_head)
        for r, li in enumerate(rows):
            res[lo + int(li)] = (o[r], x[r], z[r])
    return res


def _exercise(w, z32, amax):
    """Steer some retrieved non-greedy tokens into ranks 1..2k-1, then greedy runs."""
    p = w.params
    M = z32.shape[0]
    u = synth.uniform_stream(w.seed, synth.STREAM["exercise"], 0, 4 * M + 8)
    B = len(w.node_off) - 1
    for b in range(B):
        lo, hi = int(w.node_off[b]), int(w.node_off[b + 1])
        steered = set()
        for j in range(lo + 1, hi):
            i = lo + int(w.parent[j])
            if w.src[j] != synth.SRC_RETRIEVED or w.token[j] == amax[i]:
                # greedy continuation below a steered node
                if i in steered and u[4 * j + 2] < 0.75:
                    w.token[j] = amax[i]
                    steered.add(j)
                continue
            if i in steered and u[4 * j + 2] < 0.75:
                w.token[j] = amax[i]
                steered.add(j)
                continue
            if u[4 * j] < 0.5:
                order = _order(z32[i])
                r = 1 + min(int(u[4 * j + 1] * (2 * p.topk - 1)), 2 * p.topk - 2)
                r = min(r, z32.shape[1] - 1)
                w.token[j] = int(order[r])
                steered.add(j)


# ---------------------------------------------------------------------------
# Stochastic verification inputs
# ---------------------------------------------------------------------------

STOCH_DRAW_MARGIN = 2e-4   # relative to the residual's total mass


def _softmax_T(z, T):
    e = np.exp((z - z.max()) / T)
    return e / e.sum()


def stochastic_inputs(case: Case, temperature: float, *, seed: int = 3, with_q: bool = True, q_noise: float = 0.5):
    """Drafter distributions and uniforms for stochastic verification of ``case``.

    q at node i is softmax((z_i + noise) / T), a drafter close to the target;
    uniforms come from a seeded stream and are redrawn until every decision the
    walk can take sits >= MARGIN from its threshold (acceptance tests) or
    >= STOCH_DRAW_MARGIN of the residual mass from its bucket's edges (draws),
    so that float32 and float64 arithmetic decide alike.  Returns (q, u).
    """
    w = case.w
    z32 = case.z.astype(np.float32)
    M, V = z32.shape
    rng = np.random.default_rng(seed)
    q = None
    if with_q:
        q = np.empty((M, V), np.float32)
        for i in range(M):
            q[i] = _softmax_T(z32[i].astype(np.float64) + rng.normal(0, q_noise, V), temperature).astype(np.float32)
    u = rng.random((M, 2)).astype(np.float32)
    B = len(w.node_off) - 1
    for b in range(B):
        lo, hi = int(w.node_off[b]), int(w.node_off[b + 1])
        par = w.parent[lo:hi]
        for li in range(hi - lo):
            i = lo + li
            r = _softmax_T(z32[i].astype(np.float64), temperature)
            kids = [j for j in range(li + 1, hi - lo) if par[j] == li]
            for j in kids:
                t = int(w.token[lo + j])
                model = q is not None and int(w.src[lo + j]) != synth.SRC_RETRIEVED
                qk = q[i].astype(np.float64) if model else np.eye(1, V, t)[0]
                a = min(1.0, r[t] / qk[t]) if qk[t] > 0 else (1.0 if r[t] > 0 else 0.0)
                while abs(float(u[lo + j, 0]) - a) < MARGIN or (a >= 1.0 and u[lo + j, 0] > 1 - MARGIN):
                    u[lo + j, 0] = np.float32(rng.random())
                if float(u[lo + j, 0]) < a:
                    break                       # accepted: this node never draws
                d = np.maximum(r - qk, 0.0)
                if d.sum() > 0:
                    r = d / d.sum()
            else:
                c = np.cumsum(r)
                tot = c[-1]
                while True:
                    thr = float(u[i, 1]) * tot
                    v = int(np.searchsorted(c, thr, side="right"))
                    lo_edge = c[v - 1] if v > 0 else 0.0
                    if v < V and thr - lo_edge >= STOCH_DRAW_MARGIN * tot and c[v] - thr >= STOCH_DRAW_MARGIN * tot:
                        break
                    u[i, 1] = np.float32(rng.random())
    return q, u


def stochastic_expected(case: Case, q, u, temperature: float) -> dict:
    """The oracle's stochastic verification of every sequence of ``case``."""
    w = case.w
    e = case.expected
    z32 = case.z.astype(np.float32)
    M = z32.shape[0]
    B = len(w.node_off) - 1
    D = w.shape.max_depth
    out = dict(flags=e["flags"].copy(), sample=np.full(M, -1, np.int32), path=e["path"].copy(),
               acc_len=e["acc_len"].copy(), bonus=e["bonus"].copy(), winner_leaf=e["winner_leaf"].copy(),
               leaf_acc_len=e["leaf_acc_len"].copy())
    for b in range(B):
        lo, hi = int(w.node_off[b]), int(w.node_off[b + 1])
        if int(e["seq_status"][b]) != 0:
            continue
        r = oracle.stochastic(w.parent[lo:hi], w.token[lo:hi], w.src[lo:hi], z32[lo:hi],
                              None if q is None else q[lo:hi], u[lo:hi], temperature, D)
        f = out["flags"][lo:hi] & np.uint8(~(oracle.FLAG_ON_PATH | 32) & 0xFF)
        f |= (r["acc_bit"] * 32).astype(np.uint8)
        f[r["path"][:r["acc_len"] + 1]] |= np.uint8(oracle.FLAG_ON_PATH)
        out["flags"][lo:hi] = f
        out["sample"][lo:hi] = r["sample"]
        out["path"][b] = r["path"]
        out["acc_len"][b] = r["acc_len"]
        out["bonus"][b] = r["bonus"]
        out["winner_leaf"][b] = r["winner_leaf"]
        out["leaf_acc_len"][lo:hi] = r["leaf_acc_len"]
    return out
