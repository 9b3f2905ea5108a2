"""Pins of the oracle's per-query routing and attention (reading R14: decode
steps and the strictly causal variant) to things other than themselves: the
already pinned block routing, a per-head score formulation, the causal
structure the variant exists for, torch's dense attention and autograd.
No GPU needed.
"""

import math
from dataclasses import replace

import numpy as np
import pytest
import torch

from oracle import hga_oracle as orc
from paper_2607_15105_amd import synth


def _cfg(wl: synth.Workload) -> orc.Config:
    return orc.Config(wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.chunk_size, wl.group_size,
                      wl.query_block, wl.top_chunks, wl.top_groups, wl.sink_tokens,
                      wl.local_tokens)


def _small(**kw) -> synth.Workload:
    base = synth.Workload("small", T=512, n_q_heads=4, n_kv_heads=2, head_dim=16, dtype="fp32",
                          seed=13, q_begin=0, n_q=512, grad_begin=0, key_offset="normal",
                          top_chunks=2, top_groups=5, sink_tokens=64, local_tokens=128)
    return replace(base, **kw)


def _inputs(wl):
    return synth.queries(wl), synth.keys(wl), synth.values(wl)


def test_rows_of_equal_queries_route_like_their_block():
    """Every row of a block a copy of the block's first row: each row's own
    descriptor then equals the block descriptor, so the per-query routing of
    every row must be the (independently pinned) block routing of its block."""
    wl = _small(q_begin=192, n_q=320, top_chunks=2, top_groups=6)
    cfg = _cfg(wl)
    Q, K, _ = _inputs(wl)
    Qc = Q[wl.q_begin:].copy()
    for b in range(wl.n_q // 64):
        Qc[b * 64:(b + 1) * 64] = Qc[b * 64]
    cs, gs = orc.summaries(K, cfg)
    rb = orc.route(Qc, cs, gs, cfg, wl.q_begin, wl.n_q)
    rr = orc.route_rows(Qc, cs, gs, cfg, wl.q_begin, wl.n_q)
    for r in range(wl.n_q):
        np.testing.assert_array_equal(rr.sel_chunks[r], rb.sel_chunks[r // 64])
        np.testing.assert_array_equal(rr.sel_groups[r], rb.sel_groups[r // 64])
        np.testing.assert_array_equal(rr.n_sel_groups[r], rb.n_sel_groups[r // 64])
    assert (rb.n_sel_groups > 0).any()


def test_row_routing_matches_per_head_scores_and_a_full_sort():
    """Chunk and group scores recomputed as the mean over the G query heads of
    q . (mean key of the chunk / group), straight from the raw keys, then
    ranked by a full sort (score descending, index ascending)."""
    wl = _small(q_begin=250, n_q=70, top_chunks=3, top_groups=7)
    cfg = _cfg(wl)
    Q, K, _ = _inputs(wl)
    Qc = Q[wl.q_begin:]
    cs, gs = orc.summaries(K, cfg)
    rr = orc.route_rows(Qc, cs, gs, cfg, wl.q_begin, wl.n_q)
    G, C, g = cfg.gqa, cfg.chunk_size, cfg.group_size
    Kf = K.astype(np.float64)
    for r in range(wl.n_q):
        pos = wl.q_begin + r
        ls = max(0, (pos // 64 + 1) * 64 - wl.local_tokens)
        cands = [c for c in range(512 // C) if c * C >= wl.sink_tokens and (c + 1) * C <= ls]
        for h in range(wl.n_kv_heads):
            qs = Qc[r, h * G:(h + 1) * G].astype(np.float64)
            sc = {c: float(np.mean([q @ Kf[c * C:(c + 1) * C, h].mean(axis=0) for q in qs])) for c in cands}
            top = sorted(sorted(cands, key=lambda c: (-sc[c], c))[:wl.top_chunks])
            got = [int(c) for c in rr.sel_chunks[r, h] if c >= 0]
            assert got == top, (r, h)
            groups = [c * (C // g) + j for c in top for j in range(C // g)]
            sg = {j: float(np.mean([q @ Kf[j * g:(j + 1) * g, h].mean(axis=0) for q in qs])) for j in groups}
            topg = sorted(sorted(groups, key=lambda j: (-sg[j], j))[:wl.top_groups])
            assert [int(j) for j in rr.sel_groups[r, h, :rr.n_sel_groups[r, h]]] == topg, (r, h)


def test_row_windows_at_unaligned_positions():
    """Sink, local window and causal cut of single queries at hand-picked
    positions (Ws 64, Wl 128, B 64)."""
    cfg = orc.Config(1, 1, 8, top_chunks=0, top_groups=0, sink_tokens=64, local_tokens=128)
    cases = {
        0: [0],                                        # first token: itself only
        37: list(range(38)),                           # local [0, 64), cut at 37
        100: list(range(101)),                         # block 1: local [0, 128)
        130: list(range(64)) + list(range(64, 131)),   # block 2: local [64, 192), sink [0, 64)
        1000: list(range(64)) + list(range(896, 1001)),  # block 15: local [896, 1024)
    }
    for pos, want in cases.items():
        got = orc.routed_tokens_row(pos, np.zeros(0, np.int64), cfg)
        assert sorted(got.tolist()) == sorted(set(want)), pos
    got = orc.routed_tokens_row(1000, np.array([20, 41]), replace(cfg, group_size=8))
    assert sorted(got.tolist()) == sorted(list(range(64)) + list(range(160, 168)) + list(range(328, 336))
                                          + list(range(896, 1001)))


def test_per_query_routing_is_causal_and_block_routing_is_not():
    """The point of the variant (Sec. 6.1): changing the queries after row i
    leaves row i's routing and output unchanged under per-query routing,
    while under block routing a later query of the same block changes which
    groups an earlier one attends."""
    wl = _small(q_begin=256, n_q=256, top_chunks=2, top_groups=4)
    cfg = _cfg(wl)
    Q, K, V = _inputs(wl)
    Qc = Q[wl.q_begin:].copy()
    cs, gs = orc.summaries(K, cfg)
    i = 70                                    # row 6 of block 1 of the call
    Qp = Qc.copy()
    Qp[i + 1:] = np.random.default_rng(3).standard_normal(Qp[i + 1:].shape).astype(np.float32) * 4
    r0 = orc.route_rows(Qc, cs, gs, cfg, wl.q_begin, wl.n_q)
    r1 = orc.route_rows(Qp, cs, gs, cfg, wl.q_begin, wl.n_q)
    np.testing.assert_array_equal(r0.sel_groups[:i + 1], r1.sel_groups[:i + 1])
    O0, _ = orc.attend_rows_fwd(Qc, K, V, cfg, wl.q_begin, wl.n_q, r0.sel_groups, r0.n_sel_groups)
    O1, _ = orc.attend_rows_fwd(Qp, K, V, cfg, wl.q_begin, wl.n_q, r1.sel_groups, r1.n_sel_groups)
    np.testing.assert_array_equal(O0[:i + 1], O1[:i + 1])
    b0 = orc.route(Qc, cs, gs, cfg, wl.q_begin, wl.n_q)
    b1 = orc.route(Qp, cs, gs, cfg, wl.q_begin, wl.n_q)
    assert not np.array_equal(b0.sel_groups[i // 64], b1.sel_groups[i // 64])


def _torch_dense_rows(Q, K, V, cfg, masks):
    """Masked softmax attention by torch's own routine, float64; masks[hq] is
    [n_q, T]."""
    G = cfg.gqa
    q = torch.from_numpy(orc.widen(Q)).permute(1, 0, 2)
    k = torch.from_numpy(orc.widen(K)).permute(1, 0, 2).repeat_interleave(G, 0)
    v = torch.from_numpy(orc.widen(V)).permute(1, 0, 2).repeat_interleave(G, 0)
    m = torch.from_numpy(masks)
    o = torch.nn.functional.scaled_dot_product_attention(q, k, v, attn_mask=m, scale=cfg.scale)
    s = (q @ k.transpose(1, 2)) * cfg.scale
    lse = torch.logsumexp(s.masked_fill(~m, -math.inf), dim=-1)
    return o.permute(1, 0, 2).numpy(), lse.T.numpy()


def _row_masks(wl, r, q_begin, n_q, T):
    """[Hq, n_q, T] masks from a per-query routing, built from the window
    arithmetic directly."""
    G = wl.n_q_heads // wl.n_kv_heads
    out = np.zeros((wl.n_q_heads, n_q, T), bool)
    for row in range(n_q):
        i = q_begin + row
        ls = max(0, (i // 64 + 1) * 64 - wl.local_tokens)
        base = np.zeros(T, bool)
        base[:min(wl.sink_tokens, ls)] = True
        base[ls:i + 1] = True
        for h in range(wl.n_kv_heads):
            m = base.copy()
            for j in r.sel_groups[row, h, :r.n_sel_groups[row, h]]:
                m[j * wl.group_size:(j + 1) * wl.group_size] = True
            out[h * G:(h + 1) * G, row] = m
    return out


def test_row_attention_equals_dense_attention_under_its_mask():
    wl = _small(q_begin=200, n_q=150)
    cfg = _cfg(wl)
    Q, K, V = _inputs(wl)
    T = wl.q_begin + wl.n_q
    Qc, K, V = Q[wl.q_begin:T], K[:T], V[:T]
    cs, gs = orc.summaries(K, cfg)
    r = orc.route_rows(Qc, cs, gs, cfg, wl.q_begin, wl.n_q)
    O, lse = orc.attend_rows_fwd(Qc, K, V, cfg, wl.q_begin, wl.n_q, r.sel_groups, r.n_sel_groups)
    Od, lsed = _torch_dense_rows(Qc, K, V, cfg, _row_masks(wl, r, wl.q_begin, wl.n_q, T))
    np.testing.assert_allclose(O, Od, atol=1e-12, rtol=0)
    np.testing.assert_allclose(lse, lsed, atol=1e-12, rtol=0)


def test_row_attention_with_all_covering_budget_equals_dense_causal():
    wl = synth.WORKLOADS["tiny_fp32_1k"].with_budget(top_chunks=16, top_groups=128)
    cfg = _cfg(wl)
    Q, K, V = _inputs(wl)
    cs, gs = orc.summaries(K, cfg)
    r = orc.route_rows(Q, cs, gs, cfg, 0, wl.n_q)
    O, lse = orc.attend_rows_fwd(Q, K, V, cfg, 0, wl.n_q, r.sel_groups, r.n_sel_groups)
    causal = np.tril(np.ones((wl.T, wl.T), bool))[None]
    Od, lsed = _torch_dense_rows(Q, K, V, cfg, causal)
    np.testing.assert_allclose(O, Od, atol=1e-12, rtol=0)
    np.testing.assert_allclose(lse, lsed, atol=1e-12, rtol=0)


@pytest.mark.parametrize("grad_begin", [0, 192])
def test_row_backward_matches_torch_autograd(grad_begin):
    wl = _small(q_begin=200, n_q=120, grad_begin=grad_begin)
    cfg = _cfg(wl)
    Q, K, V = _inputs(wl)
    T = wl.q_begin + wl.n_q
    Qc, K, V = Q[wl.q_begin:T], K[:T], V[:T]
    dO = synth.grad_output(wl, wl.q_begin, T)
    cs, gs = orc.summaries(K, cfg)
    r = orc.route_rows(Qc, cs, gs, cfg, wl.q_begin, wl.n_q)
    dQ, dK, dV = orc.attend_rows_bwd(Qc, K, V, dO, cfg, wl.q_begin, wl.n_q, grad_begin,
                                     r.sel_groups, r.n_sel_groups)
    masks = torch.from_numpy(_row_masks(wl, r, wl.q_begin, wl.n_q, T))
    q = torch.tensor(orc.widen(Qc), requires_grad=True)
    k = torch.tensor(orc.widen(K), requires_grad=True)
    v = torch.tensor(orc.widen(V), requires_grad=True)
    G = cfg.gqa
    outs = []
    for hq in range(cfg.n_q_heads):
        s = (q[:, hq] @ k[:, hq // G].T) * cfg.scale
        outs.append(torch.softmax(s.masked_fill(~masks[hq], -math.inf), dim=-1) @ v[:, hq // G])
    (torch.stack(outs, dim=1) * torch.from_numpy(orc.widen(dO))).sum().backward()
    assert dK.shape[0] == T - grad_begin
    np.testing.assert_allclose(dQ, q.grad.numpy(), atol=1e-11, rtol=0)
    np.testing.assert_allclose(dK, k.grad.numpy()[grad_begin:], atol=1e-11, rtol=0)
    np.testing.assert_allclose(dV, v.grad.numpy()[grad_begin:], atol=1e-11, rtol=0)


def test_decode_one_row_at_a_time_equals_one_call():
    """Routing and attending rows one call each (decode steps) gives what one
    call over all of them gives: rows do not interact."""
    wl = _small(q_begin=300, n_q=9)
    cfg = _cfg(wl)
    Q, K, V = _inputs(wl)
    Qc = Q[wl.q_begin:wl.q_begin + wl.n_q]
    cs, gs = orc.summaries(K, cfg)
    r = orc.route_rows(Qc, cs, gs, cfg, wl.q_begin, wl.n_q)
    O, lse = orc.attend_rows_fwd(Qc, K, V, cfg, wl.q_begin, wl.n_q, r.sel_groups, r.n_sel_groups)
    for j in range(wl.n_q):
        rj = orc.route_rows(Qc[j:j + 1], cs, gs, cfg, wl.q_begin + j, 1)
        np.testing.assert_array_equal(rj.sel_groups[0], r.sel_groups[j])
        Oj, lj = orc.attend_rows_fwd(Qc[j:j + 1], K, V, cfg, wl.q_begin + j, 1, rj.sel_groups, rj.n_sel_groups)
        np.testing.assert_array_equal(Oj[0], O[j])
        np.testing.assert_array_equal(lj[0], lse[j])
