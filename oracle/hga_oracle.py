"""Plain CPU oracle for the Hierarchical Global Attention (HGA) hot path.

TEST INFRASTRUCTURE. This module is a slow, obviously-correct reference used
only to check the GPU library. Only the test suite, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py`` may import it; the product path
(the HIP library and its Python binding) never does, and shares no code with it.

What it computes, step by step (Sec. 2.1 items 1-3, Fig. 1; Sec. 2.2):

* Sec. 2.1 item 1 and Fig. 1: every completed chunk of C keys has one summary
  vector; each query block ranks those summaries and routes to its top_chunks
  winners. The sink and local windows are attended regardless of the ranking.
* Sec. 2.1 item 2: inside the winning chunks the finer g-token groups are
  ranked by their own summaries and the top_groups winners are kept.
* Sec. 2.1 item 3: softmax attention then runs over the real key and value
  rows of the kept tokens; a summary never stands in for a key or a value.
* Sec. 2.1 closing paragraph, and Sec. 2.2: the routing decision is a
  constant for differentiation; only tokens of the active segment receive
  dK/dV (truncated backpropagation), history rows receive nothing.

Arithmetic is float64 throughout. bf16 inputs (passed as uint16 bit patterns)
are widened exactly. Softmax is the two-pass textbook form (max, then sum).

Readings taken where the paper is silent (the GPU kernels take the same ones):

* R1 summary: the arithmetic mean of the keys of the chunk / group.
* R2 keys: the same K tensor that attention uses.
* R3 block score: dot product with the mean query over the block's B rows and
  the G query heads that share the kv head (equal to the mean per-query score).
* R4 granularity: one routing decision per (query block, kv head).
* R5 group scope: a global top-k over all groups of all selected chunks.
* R6 windows: sink = tokens [0, min(Ws, local_start)); local = the Wl tokens
  ending at the block end (diagonal block included), both attended in full and
  not counted in the budget; candidate chunks overlap neither window.
* R7 a chunk is routable once all its tokens precede the local window, also
  inside the current segment.
* R9 ties: score descending, then lower index first; returned sets ascending.
* R10 a budget larger than the candidate count takes every candidate.
* R11 softmax scale 1/sqrt(d) unless given; LSE in natural log.
* R13 dK/dV only for tokens >= grad_begin; history rows get no gradient.
* R15 group-summary cache (Sec. 2.1 item 2 keeps group summaries in a larger
  device cache with misses served from host memory; Table 7 reports its hit
  rate; the replacement policy is not given): whole chunks are cached (the C/g
  summaries of a chunk share a slot). A routing call reads the cache as it was
  when the call began; the chunks it chose that were not resident then enter,
  in ascending chunk order, first in first out over n_slots slots per kv head
  (the last n_slots of them when more missed).
* R14 per-query routing (decode, and the strictly causal variant of Sec. 6.1):
  a query's descriptor is the mean of its own G query-head rows (the block
  descriptor of R3 over a block of one query). Its sink window, local window
  and candidate chunks stay those of the B-block holding it (R6, R7), and it
  attends only tokens t <= its position. Its routed set then depends on its
  own row and on keys before it, never on later queries.

Pins: every function here is checked in ``tests/test_oracle_pins.py`` against
something other than itself (hand-worked fixtures, dense attention from a
library routine, torch autograd, finite differences, exhaustive top-k, the
paper's printed selection densities, a planted-recovery construction).
The choices R1, R3, R4, R5 and R14 themselves are parity unpinned: the paper
prints no routing values that could confirm them.
"""

from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class Config:
    """Problem statement of one HGA layer (Sec. 2.1; GQA head mapping q -> q // G)."""

    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    chunk_size: int = 64
    group_size: int = 8
    query_block: int = 64
    top_chunks: int = 8
    top_groups: int = 16
    sink_tokens: int = 64
    local_tokens: int = 128
    softmax_scale: float = 0.0  # <= 0 means 1/sqrt(head_dim)

    @property
    def gqa(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def scale(self) -> float:
        return self.softmax_scale if self.softmax_scale > 0 else 1.0 / math.sqrt(self.head_dim)


def widen(a: np.ndarray) -> np.ndarray:
    """Exact widening to float64: uint16 arrays are bf16 bit patterns."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


# --------------------------------------------------------------------------
# Summaries (Sec. 2.1 items 1-2: chunk and group summary vectors, reading R1)
# --------------------------------------------------------------------------

def summaries(K: np.ndarray, cfg: Config, t_end: int | None = None):
    """Mean key of every closed chunk and every complete group of K[:t_end].

    Returns (chunk_sum[Hkv, t_end // C, d], group_sum[Hkv, t_end // g, d]).
    """
    T = K.shape[0] if t_end is None else t_end
    C, g = cfg.chunk_size, cfg.group_size
    Hkv, d = cfg.n_kv_heads, cfg.head_dim
    n_chunks, n_groups = T // C, T // g
    chunk_sum = np.zeros((Hkv, n_chunks, d))
    group_sum = np.zeros((Hkv, n_groups, d))
    for c in range(n_chunks):
        keys = widen(K[c * C:(c + 1) * C])  # [C, Hkv, d]
        chunk_sum[:, c, :] = keys.sum(axis=0) / C
    for j in range(n_groups):
        keys = widen(K[j * g:(j + 1) * g])
        group_sum[:, j, :] = keys.sum(axis=0) / g
    return chunk_sum, group_sum


# --------------------------------------------------------------------------
# Routing (Sec. 2.1 items 1-2, Fig. 1; readings R3-R10)
# --------------------------------------------------------------------------

def block_descriptor(Q: np.ndarray, cfg: Config, row0: int, h: int) -> np.ndarray:
    """Mean query over the block's rows [row0, row0+B) and the G q-heads of kv head h."""
    G, B = cfg.gqa, cfg.query_block
    rows = widen(Q[row0:row0 + B, h * G:(h + 1) * G, :])  # [B, G, d]
    return rows.sum(axis=(0, 1)) / (B * G)


def windows(abs_block: int, cfg: Config):
    """(sink_end, local_start, block_end) of a query block, reading R6."""
    block_end = (abs_block + 1) * cfg.query_block
    local_start = max(0, block_end - cfg.local_tokens)
    sink_end = min(cfg.sink_tokens, local_start)
    return sink_end, local_start, block_end


def candidate_chunks(abs_block: int, cfg: Config) -> np.ndarray:
    """Closed chunks outside both windows: c*C >= Ws and (c+1)*C <= local_start (R6, R7)."""
    C = cfg.chunk_size
    _, local_start, _ = windows(abs_block, cfg)
    first = -(-cfg.sink_tokens // C)
    last = local_start // C
    return np.arange(first, last, dtype=np.int64) if last > first else np.zeros(0, np.int64)


def top_k(scores: np.ndarray, k: int) -> np.ndarray:
    """Positions of the k best scores (descending score, then lower position), ascending.

    Takes every position when k >= len(scores) (reading R10).
    """
    n = len(scores)
    if k >= n:
        return np.arange(n)
    order = np.lexsort((np.arange(n), -np.asarray(scores)))  # last key is primary
    return np.sort(order[:k])


@dataclass
class Routing:
    sel_chunks: np.ndarray    # [n_qb, Hkv, k_c] int32, ascending, -1 pad
    sel_groups: np.ndarray    # [n_qb, Hkv, k_g] int32, ascending global group ids, -1 pad
    n_sel_groups: np.ndarray  # [n_qb, Hkv] int32
    chunk_cand: list          # [n_qb][Hkv] candidate chunk ids
    chunk_scores: list        # [n_qb][Hkv] float64 scores of chunk_cand
    group_cand: list          # [n_qb][Hkv] candidate group ids
    group_scores: list        # [n_qb][Hkv] float64 scores of group_cand


def route(Q, chunk_sum, group_sum, cfg: Config, q_begin: int, n_q: int) -> Routing:
    """Two-level routing of every (query block, kv head) of rows [q_begin, q_begin+n_q)."""
    B, C, g = cfg.query_block, cfg.chunk_size, cfg.group_size
    Hkv = cfg.n_kv_heads
    n_qb = n_q // B
    kc, kg = cfg.top_chunks, cfg.top_groups
    sel_c = np.full((n_qb, Hkv, kc), -1, np.int32)
    sel_g = np.full((n_qb, Hkv, kg), -1, np.int32)
    n_sel = np.zeros((n_qb, Hkv), np.int32)
    cc, cs, gc, gs = [], [], [], []
    for b in range(n_qb):
        abs_block = q_begin // B + b
        cand = candidate_chunks(abs_block, cfg)
        rc, rs, rgc, rgs = [], [], [], []
        for h in range(Hkv):
            qbar = block_descriptor(Q, cfg, b * B, h)
            scores = chunk_sum[h, cand, :] @ qbar if len(cand) else np.zeros(0)
            chosen = cand[top_k(scores, kc)]
            groups = np.concatenate(
                [c * (C // g) + np.arange(C // g) for c in chosen]).astype(np.int64) \
                if len(chosen) else np.zeros(0, np.int64)
            gscores = group_sum[h, groups, :] @ qbar if len(groups) else np.zeros(0)
            chosen_g = groups[top_k(gscores, kg)]
            sel_c[b, h, :len(chosen)] = chosen
            sel_g[b, h, :len(chosen_g)] = chosen_g
            n_sel[b, h] = len(chosen_g)
            rc.append(cand), rs.append(scores), rgc.append(groups), rgs.append(gscores)
        cc.append(rc), cs.append(rs), gc.append(rgc), gs.append(rgs)
    return Routing(sel_c, sel_g, n_sel, cc, cs, gc, gs)


def routed_tokens(abs_block: int, groups: np.ndarray, cfg: Config) -> np.ndarray:
    """Exact token ids a block attends for one kv head: sink, selected groups, local window."""
    g = cfg.group_size
    sink_end, local_start, block_end = windows(abs_block, cfg)
    parts = [np.arange(0, sink_end)]
    parts += [np.arange(j * g, (j + 1) * g) for j in groups]
    parts.append(np.arange(local_start, block_end))
    return np.concatenate(parts).astype(np.int64)


# --------------------------------------------------------------------------
# Exact-token attention (Sec. 2.1 item 3) and its backward (Sec. 2.1, 2.2)
# --------------------------------------------------------------------------

def _block_groups(sel_groups, n_sel, b, h):
    return sel_groups[b, h, :n_sel[b, h]].astype(np.int64)


def attend_fwd(Q, K, V, cfg: Config, q_begin: int, n_q: int, sel_groups, n_sel,
               blocks=None):
    """Softmax attention of each query over its block's routed tokens t <= query.

    Returns (O[n_q, Hq, d], lse[n_q, Hq]) in float64; rows of blocks not listed
    in ``blocks`` (when given) are left as NaN.
    """
    B, G, Hkv, d = cfg.query_block, cfg.gqa, cfg.n_kv_heads, cfg.head_dim
    n_qb = n_q // B
    O = np.full((n_q, cfg.n_q_heads, d), np.nan)
    lse = np.full((n_q, cfg.n_q_heads), np.nan)
    for b in (range(n_qb) if blocks is None else blocks):
        abs_block = q_begin // B + b
        qpos = q_begin + b * B + np.arange(B)
        for h in range(Hkv):
            toks = routed_tokens(abs_block, _block_groups(sel_groups, n_sel, b, h), cfg)
            Kr, Vr = widen(K[toks, h, :]), widen(V[toks, h, :])
            allowed = toks[None, :] <= qpos[:, None]
            for hq in range(h * G, (h + 1) * G):
                q = widen(Q[b * B:(b + 1) * B, hq, :])
                s = np.where(allowed, cfg.scale * (q @ Kr.T), -np.inf)
                m = s.max(axis=1, keepdims=True)          # pass 1: row max
                p = np.exp(s - m)
                l = p.sum(axis=1, keepdims=True)          # pass 2: row sum
                O[b * B:(b + 1) * B, hq, :] = (p / l) @ Vr
                lse[b * B:(b + 1) * B, hq] = (m + np.log(l))[:, 0]
    return O, lse


def attend_bwd(Q, K, V, dO, cfg: Config, q_begin: int, n_q: int, grad_begin: int,
               sel_groups, n_sel):
    """Gradients of the routed attention; routing is a constant (no gradient).

    dQ[n_q, Hq, d] for every query; dK, dV[T_act, Hkv, d] for tokens
    [grad_begin, q_begin + n_q) only, summed over the G q-heads of each kv head.
    """
    B, G, Hkv, d = cfg.query_block, cfg.gqa, cfg.n_kv_heads, cfg.head_dim
    n_qb = n_q // B
    T_act = q_begin + n_q - grad_begin
    dQ = np.zeros((n_q, cfg.n_q_heads, d))
    dK = np.zeros((T_act, Hkv, d))
    dV = np.zeros((T_act, Hkv, d))
    for b in range(n_qb):
        abs_block = q_begin // B + b
        qpos = q_begin + b * B + np.arange(B)
        for h in range(Hkv):
            toks = routed_tokens(abs_block, _block_groups(sel_groups, n_sel, b, h), cfg)
            Kr, Vr = widen(K[toks, h, :]), widen(V[toks, h, :])
            allowed = toks[None, :] <= qpos[:, None]
            dKr = np.zeros_like(Kr)
            dVr = np.zeros_like(Vr)
            for hq in range(h * G, (h + 1) * G):
                rows = slice(b * B, (b + 1) * B)
                q, do = widen(Q[rows, hq, :]), widen(dO[rows, hq, :])
                s = np.where(allowed, cfg.scale * (q @ Kr.T), -np.inf)
                m = s.max(axis=1, keepdims=True)
                p = np.exp(s - m)
                P = p / p.sum(axis=1, keepdims=True)
                dP = do @ Vr.T
                Dv = (P * dP).sum(axis=1, keepdims=True)
                dS = P * (dP - Dv)
                dQ[rows, hq, :] = cfg.scale * (dS @ Kr)
                dKr += cfg.scale * (dS.T @ q)
                dVr += P.T @ do
            active = toks >= grad_begin
            np.add.at(dK[:, h, :], toks[active] - grad_begin, dKr[active])
            np.add.at(dV[:, h, :], toks[active] - grad_begin, dVr[active])
    return dQ, dK, dV


# --------------------------------------------------------------------------
# Per-query routing (reading R14): decode-time routing (Sec. 1, last result;
# Sec. 4.6 and 7 mention routed generation) and the strictly causal variant
# the paper leaves open (Sec. 6.1)
# --------------------------------------------------------------------------

def query_descriptor(Q: np.ndarray, cfg: Config, row: int, h: int) -> np.ndarray:
    """Mean of one query row's G query heads of kv head h (R3 with B = 1)."""
    G = cfg.gqa
    return widen(Q[row, h * G:(h + 1) * G, :]).sum(axis=0) / G


def route_rows(Q, chunk_sum, group_sum, cfg: Config, q_begin: int, n_q: int) -> Routing:
    """Two-level routing of every (query row, kv head) of rows [q_begin, q_begin+n_q).

    q_begin and n_q are arbitrary (a decode step is n_q = 1). Each row takes
    the candidate chunks of the block holding it and its own descriptor; the
    outputs are indexed [row, kv head, k] like the block routing's [block,
    kv head, k].
    """
    B, C, g = cfg.query_block, cfg.chunk_size, cfg.group_size
    Hkv = cfg.n_kv_heads
    kc, kg = cfg.top_chunks, cfg.top_groups
    sel_c = np.full((n_q, Hkv, kc), -1, np.int32)
    sel_g = np.full((n_q, Hkv, kg), -1, np.int32)
    n_sel = np.zeros((n_q, Hkv), np.int32)
    cc, cs, gc, gs = [], [], [], []
    for r in range(n_q):
        cand = candidate_chunks((q_begin + r) // B, cfg)
        rc, rs, rgc, rgs = [], [], [], []
        for h in range(Hkv):
            qd = query_descriptor(Q, cfg, r, h)
            scores = chunk_sum[h, cand, :] @ qd if len(cand) else np.zeros(0)
            chosen = cand[top_k(scores, kc)]
            groups = np.concatenate(
                [c * (C // g) + np.arange(C // g) for c in chosen]).astype(np.int64) \
                if len(chosen) else np.zeros(0, np.int64)
            gscores = group_sum[h, groups, :] @ qd if len(groups) else np.zeros(0)
            chosen_g = groups[top_k(gscores, kg)]
            sel_c[r, h, :len(chosen)] = chosen
            sel_g[r, h, :len(chosen_g)] = chosen_g
            n_sel[r, h] = len(chosen_g)
            rc.append(cand), rs.append(scores), rgc.append(groups), rgs.append(gscores)
        cc.append(rc), cs.append(rs), gc.append(rgc), gs.append(rgs)
    return Routing(sel_c, sel_g, n_sel, cc, cs, gc, gs)


def routed_tokens_row(pos: int, groups: np.ndarray, cfg: Config) -> np.ndarray:
    """Tokens a query at position pos attends for one kv head (R14): its
    block's sink window, its selected groups, and its block's local window up
    to and including pos."""
    g = cfg.group_size
    sink_end, local_start, _ = windows(pos // cfg.query_block, cfg)
    parts = [np.arange(0, sink_end)]
    parts += [np.arange(j * g, (j + 1) * g) for j in groups]
    parts.append(np.arange(local_start, pos + 1))
    return np.concatenate(parts).astype(np.int64)


def attend_rows_fwd(Q, K, V, cfg: Config, q_begin: int, n_q: int, sel_groups, n_sel):
    """Softmax attention of each query row over its own routed tokens.

    Returns (O[n_q, Hq, d], lse[n_q, Hq]) in float64.
    """
    G, Hkv, d = cfg.gqa, cfg.n_kv_heads, cfg.head_dim
    O = np.zeros((n_q, cfg.n_q_heads, d))
    lse = np.zeros((n_q, cfg.n_q_heads))
    for r in range(n_q):
        for h in range(Hkv):
            toks = routed_tokens_row(q_begin + r, _block_groups(sel_groups, n_sel, r, h), cfg)
            Kr, Vr = widen(K[toks, h, :]), widen(V[toks, h, :])
            for hq in range(h * G, (h + 1) * G):
                s = cfg.scale * (Kr @ widen(Q[r, hq, :]))
                m = s.max()                                # pass 1: max
                p = np.exp(s - m)
                l = p.sum()                                # pass 2: sum
                O[r, hq, :] = (p / l) @ Vr
                lse[r, hq] = m + np.log(l)
    return O, lse


def attend_rows_bwd(Q, K, V, dO, cfg: Config, q_begin: int, n_q: int, grad_begin: int,
                    sel_groups, n_sel):
    """Gradients of attend_rows_fwd with the routing held constant: dQ for
    every row, dK / dV for tokens [grad_begin, q_begin + n_q) summed over the
    G query heads of each kv head (R13)."""
    G, Hkv, d = cfg.gqa, cfg.n_kv_heads, cfg.head_dim
    T_act = q_begin + n_q - grad_begin
    dQ = np.zeros((n_q, cfg.n_q_heads, d))
    dK = np.zeros((T_act, Hkv, d))
    dV = np.zeros((T_act, Hkv, d))
    for r in range(n_q):
        for h in range(Hkv):
            toks = routed_tokens_row(q_begin + r, _block_groups(sel_groups, n_sel, r, h), cfg)
            Kr, Vr = widen(K[toks, h, :]), widen(V[toks, h, :])
            dKr = np.zeros_like(Kr)
            dVr = np.zeros_like(Vr)
            for hq in range(h * G, (h + 1) * G):
                q, do = widen(Q[r, hq, :]), widen(dO[r, hq, :])
                s = cfg.scale * (Kr @ q)
                p = np.exp(s - s.max())
                P = p / p.sum()
                dP = Vr @ do
                dS = P * (dP - (P * dP).sum())
                dQ[r, hq, :] = cfg.scale * (dS @ Kr)
                dKr += cfg.scale * np.outer(dS, q)
                dVr += np.outer(P, do)
            active = toks >= grad_begin
            np.add.at(dK[:, h, :], toks[active] - grad_begin, dKr[active])
            np.add.at(dV[:, h, :], toks[active] - grad_begin, dVr[active])
    return dQ, dK, dV


# --------------------------------------------------------------------------
# Group-summary cache (reading R15; the hit statistic of Table 7)
# --------------------------------------------------------------------------

def group_cache_hits(calls, n_kv_heads: int, n_slots: int):
    """Hit flags of a sequence of routing calls against the bounded cache.

    calls: list of sel_chunks arrays [n_qb, Hkv, k_c] (ascending, -1 pad), in
    call order. Returns one int array per call, shaped like its sel_chunks:
    1 where the chunk was resident when the call began, 0 where it was not,
    -1 where no chunk was chosen.
    """
    resident = [dict() for _ in range(n_kv_heads)]   # chunk -> slot
    slots = [[None] * n_slots for _ in range(n_kv_heads)]
    cursor = [0] * n_kv_heads
    out = []
    for sel in calls:
        sel = np.asarray(sel)
        hits = np.full(sel.shape, -1, np.int32)
        for h in range(n_kv_heads):
            chosen = sel[:, h, :]
            for b in range(chosen.shape[0]):
                for r in range(chosen.shape[1]):
                    if chosen[b, r] >= 0:
                        hits[b, h, r] = 1 if int(chosen[b, r]) in resident[h] else 0
            missed = sorted({int(c) for c in chosen[hits[:, h, :] == 0]})
            keep = missed[-n_slots:] if missed else []
            for k, c in enumerate(keep):
                slot = (cursor[h] + k) % n_slots
                old = slots[h][slot]
                if old is not None:
                    del resident[h][old]
                slots[h][slot] = c
                resident[h][c] = slot
            cursor[h] = (cursor[h] + len(keep)) % n_slots
        out.append(hits)
    return out


# --------------------------------------------------------------------------
# Selection density (the statistic of Tables 1, 4, 5 and 7)
# --------------------------------------------------------------------------

def selection_density(routing: Routing, cfg: Config, q_begin: int, n_q: int, h: int = 0) -> float:
    """Attended (query, key) pairs over causal pairs, for one kv head."""
    B = cfg.query_block
    attended = causal = 0
    for b in range(n_q // B):
        abs_block = q_begin // B + b
        toks = routed_tokens(abs_block, _block_groups(routing.sel_groups, routing.n_sel_groups, b, h), cfg)
        for i in range(q_begin + b * B, q_begin + (b + 1) * B):
            attended += int(np.count_nonzero(toks <= i))
            causal += i + 1
    return attended / causal
