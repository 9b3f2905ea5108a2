"""Shared helpers of the GPU parity tests: run the HIP path and the oracle on
the same seeded inputs, and compare routing with near-tie classification.

Routing rule: GPU index sets must equal the oracle's, except where a differing
index has an oracle float64 score within 1e-5 relative of the k-th selected
score (floor 1e-3 of the largest |score|); such near-ties are counted and the
outputs are then compared against the oracle run on the GPU's index set.
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np
import torch

from oracle import hga_oracle as orc
from paper_2607_15105_amd import hga, synth

NEAR_TIE_REL = 1e-5
TOL = {"bf16": 2e-2, "fp32": 1e-4}       # O, dQ, dK, dV max-abs
LSE_TOL = {"bf16": 1e-3, "fp32": 1e-4}


def cfg_of(wl: synth.Workload) -> orc.Config:
    return orc.Config(wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.chunk_size, wl.group_size,
                      wl.query_block, wl.top_chunks, wl.top_groups, wl.sink_tokens,
                      wl.local_tokens)


def hcfg_of(wl: synth.Workload) -> hga.Config:
    return hga.make_config(wl.n_q_heads, wl.n_kv_heads, wl.head_dim, chunk_size=wl.chunk_size,
                           group_size=wl.group_size, query_block=wl.query_block,
                           top_chunks=wl.top_chunks, top_groups=wl.top_groups,
                           sink_tokens=wl.sink_tokens, local_tokens=wl.local_tokens,
                           dtype=torch.bfloat16 if wl.dtype == "bf16" else torch.float32)


def to_dev(x: np.ndarray, device="cuda") -> torch.Tensor:
    """uint16 (bf16 bits) -> bfloat16 tensor; float32 -> float32 tensor."""
    if x.dtype == np.uint16:
        return torch.from_numpy(x.view(np.int16).copy()).to(device).view(torch.bfloat16)
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(device)


def to_np(t: torch.Tensor) -> np.ndarray:
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.cpu().numpy()


@dataclass
class Inputs:
    Q: np.ndarray      # rows [q_begin, q_begin + n_q)
    K: np.ndarray      # rows [0, q_begin + n_q)
    V: np.ndarray
    dO: np.ndarray | None


def make_inputs(wl: synth.Workload, backward: bool | None = None) -> Inputs:
    end = wl.q_begin + wl.n_q
    bw = wl.backward if backward is None else backward
    return Inputs(synth.queries(wl, wl.q_begin, end), synth.keys(wl, 0, end),
                  synth.values(wl, 0, end),
                  synth.grad_output(wl, wl.q_begin, end) if bw else None)


@dataclass
class GpuRun:
    chunk_sum: torch.Tensor
    group_sum: torch.Tensor
    sel_chunks: np.ndarray
    sel_groups: np.ndarray
    n_sel: np.ndarray
    O: torch.Tensor
    lse: torch.Tensor
    dQ: torch.Tensor | None = None
    dK: torch.Tensor | None = None
    dV: torch.Tensor | None = None
    o32: torch.Tensor | None = None


def gpu_run(wl: synth.Workload, inp: Inputs, backward: bool, segment: int = 0,
            fused: bool = False, bwd_kv_parts: int = 0) -> GpuRun:
    """Summaries (optionally built segment by segment), route, fwd, [bwd] through the C ABI;
    with `fused` routing and forward go through hga_route_attend_fwd; `bwd_kv_parts`
    is the backward's dK/dV partition (0 = the library's choice)."""
    hc = hcfg_of(wl)
    hc.bwd_kv_parts = bwd_kv_parts
    Q, K, V = to_dev(inp.Q), to_dev(inp.K), to_dev(inp.V)
    end = wl.q_begin + wl.n_q
    cs, gs = hga.alloc_summaries(hc, end)
    step = segment or end
    for t0 in range(0, end, step):
        hga.build_summaries(hc, K, t0, min(end, t0 + step), cs, gs)
    rb = hga.alloc_route(hc, wl.q_begin, wl.n_q)
    O = torch.empty_like(Q)
    lse = torch.empty(wl.n_q, wl.n_q_heads, device="cuda")
    o32 = torch.empty(wl.n_q, wl.n_q_heads, wl.head_dim, device="cuda") if backward else None
    if fused:
        hga.route_attend_fwd(hc, Q, K, V, wl.q_begin, cs, gs, rb.sel_chunks, rb.sel_groups,
                             rb.n_sel_groups, O, lse, rb.workspace, o32)
    else:
        hga.route(hc, Q, wl.q_begin, cs, gs, rb.sel_chunks, rb.sel_groups, rb.n_sel_groups,
                  rb.workspace)
        hga.attend_fwd(hc, Q, K, V, wl.q_begin, rb.sel_groups, rb.n_sel_groups, O, lse, o32)
    run = GpuRun(cs, gs, rb.sel_chunks.cpu().numpy(), rb.sel_groups.cpu().numpy(),
                 rb.n_sel_groups.cpu().numpy(), O, lse)
    if backward:
        dO = to_dev(inp.dO)
        n_act = end - wl.grad_begin
        run.dQ = torch.empty(wl.n_q, wl.n_q_heads, wl.head_dim, device="cuda")
        run.dK = torch.empty(n_act, wl.n_kv_heads, wl.head_dim, device="cuda")
        run.dV = torch.empty_like(run.dK)
        ws = torch.empty(hga.workspace_size(hc, hga.OP_BWD, wl.q_begin, wl.n_q, wl.grad_begin), dtype=torch.uint8,
                         device="cuda")
        hga.attend_bwd(hc, Q, K, V, O, dO, lse, wl.q_begin, wl.grad_begin, rb.sel_groups,
                       rb.n_sel_groups, run.dQ, run.dK, run.dV, ws, o32)
        run.o32 = o32
    torch.cuda.synchronize()
    return run


@dataclass
class RouteReport:
    exact: int = 0         # (block, head) pairs identical at both levels
    near_ties: int = 0     # pairs that differ only at near-ties
    mismatches: int = 0    # pairs that differ beyond the near-tie band
    detail: list | None = None


def _near_tie_set_ok(cand, scores, k, got, want) -> bool:
    """Does every index in the symmetric difference of two top-k sets sit at a near-tie?"""
    diff = set(got) ^ set(want)
    if not diff:
        return True
    if len(got) != len(want):
        return False
    pos = {c: i for i, c in enumerate(cand)}
    if any(x not in pos for x in diff):
        return False
    sk = min(scores[pos[c]] for c in want)  # oracle's k-th score
    floor = 1e-3 * float(np.max(np.abs(scores))) if len(scores) else 0.0
    band = NEAR_TIE_REL * max(abs(sk), floor)
    return all(abs(scores[pos[x]] - sk) <= band for x in diff)


def compare_routing(wl: synth.Workload, run: GpuRun, ro: orc.Routing, group_sum: np.ndarray,
                    Q: np.ndarray, rows: bool = False) -> RouteReport:
    """Bit-exact comparison, with near-tie classification, of GPU vs oracle
    routing; per block, or per query row with `rows` (per-query routing)."""
    cfg = cfg_of(wl)
    rep = RouteReport(detail=[])
    C, g = cfg.chunk_size, cfg.group_size
    for b in range(wl.n_q if rows else wl.n_q // 64):
        for h in range(cfg.n_kv_heads):
            gc = [int(c) for c in run.sel_chunks[b, h, :wl.top_chunks] if c >= 0] if wl.top_chunks else []
            oc = [int(c) for c in ro.sel_chunks[b, h] if c >= 0]
            n = int(run.n_sel[b, h])
            gg = [int(j) for j in run.sel_groups[b, h, :n]] if wl.top_groups else []
            og = [int(j) for j in ro.sel_groups[b, h, :ro.n_sel_groups[b, h]]]
            sorted_ok = gc == sorted(gc) and gg == sorted(gg) and \
                all(c == -1 for c in run.sel_chunks[b, h, len(gc):wl.top_chunks]) and \
                all(j == -1 for j in run.sel_groups[b, h, n:wl.top_groups])
            if gc == oc and gg == og and sorted_ok:
                rep.exact += 1
                continue
            ok = sorted_ok and _near_tie_set_ok(list(ro.chunk_cand[b][h]), ro.chunk_scores[b][h],
                                                wl.top_chunks, gc, oc)
            if ok:
                # group level judged against the oracle's selection over the GPU's chunks
                qbar = orc.query_descriptor(Q, cfg, b, h) if rows else orc.block_descriptor(Q, cfg, b * 64, h)
                groups = np.array([c * (C // g) + j for c in gc for j in range(C // g)], np.int64)
                gsc = group_sum[h, groups] @ qbar if len(groups) else np.zeros(0)
                want = [int(x) for x in groups[orc.top_k(gsc, wl.top_groups)]]
                ok = _near_tie_set_ok(list(groups), gsc, wl.top_groups, gg, want)
            if ok:
                rep.near_ties += 1
            else:
                rep.mismatches += 1
                if len(rep.detail) < 5:
                    rep.detail.append((b, h, gc, oc, gg, og))
    return rep


def max_abs(gpu: torch.Tensor, ref: np.ndarray) -> float:
    g = gpu.float().cpu().numpy().astype(np.float64)
    return float(np.max(np.abs(g - ref))) if g.size else 0.0
