"""GPU parity: the HIP library (through its C ABI) against the CPU oracle.

Bars: summaries bit-exact for bf16 inputs (one rounding of an exact mean) and
within one float32 ulp for fp32 inputs; routing indices bit-exact up to counted
near-ties; O, dQ, dK, dV within 2e-2 max-abs (bf16 inputs, fp32 accumulation)
or 1e-4 (fp32 inputs).
"""

import sys
from dataclasses import replace

import numpy as np
import pytest
import torch

from oracle import hga_oracle as orc
from paper_2607_15105_amd import hga, synth
from tests import parity as P

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    hga.lib()


def _oracle(wl, inp, backward, routing_from=None):
    cfg = P.cfg_of(wl)
    end = wl.q_begin + wl.n_q
    cs, gs = orc.summaries(inp.K, cfg, end)
    ro = orc.route(inp.Q, cs, gs, cfg, wl.q_begin, wl.n_q)
    sel, n = (ro.sel_groups, ro.n_sel_groups) if routing_from is None else routing_from
    O, lse = orc.attend_fwd(inp.Q, inp.K, inp.V, cfg, wl.q_begin, wl.n_q, sel, n)
    grads = None
    if backward:
        grads = orc.attend_bwd(inp.Q, inp.K, inp.V, inp.dO, cfg, wl.q_begin, wl.n_q,
                               wl.grad_begin, sel, n)
    return cs, gs, ro, O, lse, grads


def _check_summaries(wl, run, cs, gs):
    tol_ulp = 0 if wl.dtype == "bf16" else 1
    for got, ref in ((run.chunk_sum, cs), (run.group_sum, gs)):
        g = hga.summary_rows(got).cpu().numpy()[:, :ref.shape[1]]
        r = ref.astype(np.float32)
        ulps = np.abs(g.view(np.int32).astype(np.int64) - r.view(np.int32).astype(np.int64))
        assert int(ulps.max()) <= tol_ulp, f"summary off by {ulps.max()} ulp"


def _full_check(wl, backward=None, segment=0, expect_exact_routing=False, fused=False, bwd_kv_parts=0):
    backward = wl.backward if backward is None else backward
    say(f"[parity] {wl.name} T={wl.q_begin + wl.n_q} q_begin={wl.q_begin} n_q={wl.n_q} "
        f"g={wl.group_size} kc={wl.top_chunks} kg={wl.top_groups} bwd={backward} fused={fused} "
        f"bwd_kv_parts={bwd_kv_parts}")
    inp = P.make_inputs(wl, backward)
    run = P.gpu_run(wl, inp, backward, segment, fused, bwd_kv_parts)
    cs, gs, ro, _, _, _ = _oracle(wl, inp, False)
    _check_summaries(wl, run, cs, gs)
    rep = P.compare_routing(wl, run, ro, gs, inp.Q)
    say(f"[parity] routing exact={rep.exact} near_ties={rep.near_ties} mismatches={rep.mismatches}")
    assert rep.mismatches == 0, rep.detail
    if expect_exact_routing:
        assert rep.near_ties == 0
    # outputs against the oracle run on the GPU's (validated) index sets
    sel, n = run.sel_groups[:, :, :max(wl.top_groups, 1)], run.n_sel
    if wl.top_groups == 0:
        sel = np.full(sel.shape, -1, np.int32)
    cfg = P.cfg_of(wl)
    O, lse = orc.attend_fwd(inp.Q, inp.K, inp.V, cfg, wl.q_begin, wl.n_q, sel, n)
    tol = P.TOL[wl.dtype]
    eo = P.max_abs(run.O, O)
    el = P.max_abs(run.lse, lse)
    say(f"[parity] O max-abs {eo:.3g}  LSE max-abs {el:.3g}")
    assert eo <= tol and el <= P.LSE_TOL[wl.dtype]
    if backward:
        dQ, dK, dV = orc.attend_bwd(inp.Q, inp.K, inp.V, inp.dO, cfg, wl.q_begin, wl.n_q,
                                    wl.grad_begin, sel, n)
        eq, ek, ev = P.max_abs(run.dQ, dQ), P.max_abs(run.dK, dK), P.max_abs(run.dV, dV)
        say(f"[parity] dQ {eq:.3g} dK {ek:.3g} dV {ev:.3g}")
        assert eq <= tol and ek <= tol and ev <= tol
    return run, inp


# ------------------------------------------------------------------ workloads

def test_tiny_fp32_forward():
    _full_check(synth.WORKLOADS["tiny_fp32_1k"], expect_exact_routing=True)


def test_tiny_fp32_all_covering_equals_dense_causal():
    wl = synth.WORKLOADS["tiny_fp32_1k"].with_budget(top_chunks=16, top_groups=64, group_size=16)
    run, inp = _full_check(wl)
    q = torch.from_numpy(inp.Q.astype(np.float64)).permute(1, 0, 2)
    k = torch.from_numpy(inp.K.astype(np.float64)).permute(1, 0, 2)
    v = torch.from_numpy(inp.V.astype(np.float64)).permute(1, 0, 2)
    dense = torch.nn.functional.scaled_dot_product_attention(q, k, v, is_causal=True)
    assert P.max_abs(run.O, dense.permute(1, 0, 2).numpy()) <= 1e-4


def test_tiny_fp32_backward():
    wl = replace(synth.WORKLOADS["tiny_fp32_1k"], backward=True, q_begin=512, n_q=512,
                 grad_begin=256, n_q_heads=2)
    _full_check(wl)


def test_qwen3_8b_2k_forward_backward():
    _full_check(synth.WORKLOADS["qwen3_8b_2k"])


def test_qwen3_8b_16k_last_segment():
    """Summaries built segment by segment; history detached (grad_begin = segment start)."""
    _full_check(synth.WORKLOADS["qwen3_8b_16k_seg1k"], segment=1024)


@pytest.mark.parametrize("seg", [0, 3])
def test_qwen3_8b_16k_short_history_segment(seg):
    """Segments whose first block has fewer than 6 * top_chunks history chunks:
    the dK/dV work is split over two query-head subsets and summed by a
    further kernel (the workspace then holds more than D)."""
    wl = synth.WORKLOADS["qwen3_8b_16k_seg1k"]
    t0 = seg * 1024
    wl = replace(wl, T=t0 + 1024, q_begin=t0, grad_begin=t0)
    hc = P.hcfg_of(wl)
    assert hga.workspace_size(hc, hga.OP_BWD, t0, 1024, t0) > 1024 * 32 * 4
    _full_check(wl, segment=1024)


@pytest.mark.parametrize("seg,parts", [(15, 2), (0, 1)])
def test_qwen3_8b_16k_caller_chosen_dkdv_partition(seg, parts):
    """The caller's dK/dV partition against the library's choice: two
    query-head subsets on the last segment (where the library would not
    split), one item per (chunk, kv head) on segment 0 (where it would)."""
    wl = synth.WORKLOADS["qwen3_8b_16k_seg1k"]
    t0 = seg * 1024
    wl = replace(wl, T=t0 + 1024, q_begin=t0, grad_begin=t0)
    hc = P.hcfg_of(wl)
    hc.bwd_kv_parts = parts
    split = hga.workspace_size(hc, hga.OP_BWD, t0, 1024, t0) > 1024 * 32 * 4
    assert split == (parts == 2)
    _full_check(wl, segment=1024, bwd_kv_parts=parts)


@pytest.mark.parametrize("seg", [15, 2, 1, 0])
def test_fused_route_attend_16k_segment(seg):
    """Routing and forward of a 1,024-token segment as one launch
    (hga_route_attend_fwd), then the backward on its routing tables."""
    wl = synth.WORKLOADS["qwen3_8b_16k_seg1k"]
    t0 = seg * 1024
    wl = replace(wl, T=t0 + 1024, q_begin=t0, grad_begin=t0)
    _full_check(wl, segment=1024, fused=True)


def test_fused_route_attend_fp32_two_heads():
    wl = replace(synth.WORKLOADS["tiny_fp32_1k"], backward=True, q_begin=512, n_q=512,
                 grad_begin=256, n_q_heads=2)
    _full_check(wl, fused=True)


@pytest.mark.parametrize("name,q_begin,n_q", [("qwen3_8b_16k_seg1k", 15360, 1024),
                                              ("qwen3_8b_16k_seg1k", 0, 1024),
                                              ("qwen3_8b_32k_sweep", 31744, 1024),
                                              ("qwen3_8b_2k", 0, 2048),
                                              ("tiny_fp32_1k", 0, 1024)])
def test_fused_route_attend_equals_two_calls(name, q_begin, n_q):
    """hga_route_attend_fwd gives bit for bit the routing tables, O, LSE and
    float32 O of hga_route followed by hga_attend_fwd, fused or not (the
    2K call and the one-head fp32 call take the two-kernel path)."""
    wl = replace(synth.WORKLOADS[name], q_begin=q_begin, n_q=n_q, grad_begin=q_begin, T=q_begin + n_q)
    say(f"[parity] fused vs two calls: {name} q_begin={q_begin} n_q={n_q}")
    inp = P.make_inputs(wl, True)
    a = P.gpu_run(wl, inp, True, 1024 if n_q == 1024 and q_begin else 0, fused=False)
    b = P.gpu_run(wl, inp, True, 1024 if n_q == 1024 and q_begin else 0, fused=True)
    np.testing.assert_array_equal(a.sel_chunks, b.sel_chunks)
    np.testing.assert_array_equal(a.sel_groups, b.sel_groups)
    np.testing.assert_array_equal(a.n_sel, b.n_sel)
    for x, y in ((a.O, b.O), (a.lse, b.lse), (a.o32, b.o32), (a.dQ, b.dQ), (a.dK, b.dK)):
        assert torch.equal(x, y)


def test_routing_with_several_blocks_per_workgroup():
    """Every query of a 32K context in one call: 4,096 (block, kv head) pairs
    and at most 507 candidate chunks, so each routing workgroup serves two
    blocks with their whole candidate lists in one score table."""
    wl = replace(synth.WORKLOADS["qwen3_8b_32k_sweep"], q_begin=0, n_q=32768, grad_begin=0,
                 backward=False)
    cfg = P.cfg_of(wl)
    inp = P.make_inputs(wl, False)
    run = P.gpu_run(wl, inp, False)
    cs, gs = orc.summaries(inp.K, cfg)
    _check_summaries(wl, run, cs, gs)
    ro = orc.route(inp.Q, cs, gs, cfg, 0, wl.n_q)
    rep = P.compare_routing(wl, run, ro, gs, inp.Q)
    say(f"[32k all] routing exact={rep.exact} near_ties={rep.near_ties} mismatches={rep.mismatches}")
    assert rep.mismatches == 0, rep.detail
    blocks = list(range(0, wl.n_q // 64, 37))
    O, lse = orc.attend_fwd(inp.Q, inp.K, inp.V, cfg, 0, wl.n_q, run.sel_groups, run.n_sel, blocks=blocks)
    rows = np.concatenate([np.arange(b * 64, (b + 1) * 64) for b in blocks])
    assert P.max_abs(run.O[rows], O[rows]) <= P.TOL["bf16"]


def test_routing_in_rounds_with_tie_copies():
    """Every query of a 64K context: 8,192 (block, kv head) pairs with up to
    1,019 candidate chunks, so each routing workgroup serves four blocks and
    scores and selects their chunks in rounds of 512, keeping a running
    selection. 64 chunks are bit-identical copies of others: exact ties,
    some across rounds, that must go to the lower chunk index."""
    wl = replace(synth.WORKLOADS["qwen3_8b_32k_sweep"], T=65536, q_begin=0, n_q=65536, grad_begin=0,
                 tie_copies=64, backward=False)
    cfg = P.cfg_of(wl)
    inp = P.make_inputs(wl, False)
    run = P.gpu_run(wl, inp, False)
    cs, gs = orc.summaries(inp.K, cfg)
    _check_summaries(wl, run, cs, gs)
    ro = orc.route(inp.Q, cs, gs, cfg, 0, wl.n_q)
    rep = P.compare_routing(wl, run, ro, gs, inp.Q)
    say(f"[64k rounds] routing exact={rep.exact} near_ties={rep.near_ties} mismatches={rep.mismatches}")
    # an exact tie the kernel broke the other way would count as a near-tie;
    # distinct float64 scores within rounding of each other do not occur here
    assert rep.mismatches == 0 and rep.near_ties == 0, rep.detail
    blocks = list(range(5, wl.n_q // 64, 97))
    O, lse = orc.attend_fwd(inp.Q, inp.K, inp.V, cfg, 0, wl.n_q, run.sel_groups, run.n_sel, blocks=blocks)
    rows = np.concatenate([np.arange(b * 64, (b + 1) * 64) for b in blocks])
    assert P.max_abs(run.O[rows], O[rows]) <= P.TOL["bf16"]


@pytest.mark.parametrize("g,kc,kg", synth.SWEEP)
def test_32k_sweep_last_segment(g, kc, kg):
    """Every (group size, top chunks, top groups) point the benchmark times."""
    wl = synth.WORKLOADS["qwen3_8b_32k_sweep"].with_budget(group_size=g, top_chunks=kc,
                                                           top_groups=kg)
    _full_check(wl)


def test_routing_beyond_8192_chunks_in_rounds():
    """A 1,048,576-token context (16,384 chunks): the call's 16 blocks have up
    to 16,379 candidate chunks each, more than a one-block workgroup's LDS
    holds, so they are scored and selected in rounds of 512 with a running
    selection (two blocks per workgroup). Summaries, routing, O, LSE, dQ, dK
    and dV against the oracle; the fused entry point (which then runs the
    two calls) gives the same routing and O bit for bit."""
    T = 1 << 20
    wl = synth.Workload("long_1m", T=T, n_q_heads=4, n_kv_heads=1, head_dim=64, dtype="bf16", seed=11,
                        q_begin=T - 1024, n_q=1024, grad_begin=T - 1024, key_offset="normal")
    run, inp = _full_check(wl)
    fused = P.gpu_run(wl, inp, True, fused=True)  # with the float32 O, as the run above
    assert np.array_equal(fused.sel_chunks, run.sel_chunks) and np.array_equal(fused.sel_groups, run.sel_groups)
    for k in ("O", "lse", "dQ", "dK", "dV"):
        assert torch.equal(getattr(fused, k), getattr(run, k)), k


def test_exact_tie_copies_route_to_lower_index():
    wl = replace(synth.WORKLOADS["qwen3_8b_32k_sweep"], T=8192, q_begin=6144, n_q=2048,
                 grad_begin=6144, tie_copies=32, backward=False)
    _full_check(wl, expect_exact_routing=False)


# ------------------------------------------------------------------ edge cases

@pytest.mark.parametrize("kw", [
    dict(top_chunks=0),                      # sink + local only
    dict(top_groups=0),                      # chunks chosen, no groups opened
    dict(q_begin=0, n_q=64, grad_begin=0),   # a single block, nothing routable
    dict(top_chunks=64, top_groups=64, group_size=4),  # budget above the candidates
    dict(group_size=64, top_groups=3),       # whole-chunk groups
    dict(head_dim=64),
    dict(n_q_heads=8, n_kv_heads=8),         # no GQA
    dict(n_q_heads=16, n_kv_heads=8),        # GQA 2:1
    dict(n_q_heads=32, n_kv_heads=4),        # GQA 8:1
    dict(sink_tokens=0, local_tokens=64),
    dict(top_groups=13, group_size=8),       # ragged last tile
])
def test_edge_cases(kw):
    base = synth.Workload("edge", T=2048, n_q_heads=8, n_kv_heads=2, head_dim=128, dtype="bf16",
                          seed=21, q_begin=1024, n_q=1024, grad_begin=512, key_offset="normal")
    _full_check(replace(base, **kw))


def test_poisoned_unrouted_rows_do_not_reach_the_output():
    wl = synth.Workload("poison", T=2048, n_q_heads=8, n_kv_heads=2, head_dim=128, dtype="bf16",
                        seed=22, q_begin=1024, n_q=1024, grad_begin=1024, key_offset="normal",
                        backward=False)
    inp = P.make_inputs(wl)
    run = P.gpu_run(wl, inp, False)
    cfg = P.cfg_of(wl)
    K, V = inp.K.copy(), inp.V.copy()
    for h in range(wl.n_kv_heads):
        used = np.zeros(wl.T, bool)
        for b in range(wl.n_q // 64):
            used[orc.routed_tokens(wl.q_begin // 64 + b, run.sel_groups[b, h, :run.n_sel[b, h]], cfg)] = True
        K[~used, h] = 0x7FC0  # bf16 NaN
        V[~used, h] = 0x7FC0
    hc = P.hcfg_of(wl)
    Qd, Kd, Vd = P.to_dev(inp.Q), P.to_dev(K), P.to_dev(V)
    O = torch.empty_like(Qd)
    lse = torch.empty(wl.n_q, wl.n_q_heads, device="cuda")
    sg = torch.from_numpy(run.sel_groups).cuda()
    ns = torch.from_numpy(run.n_sel).cuda()
    hga.attend_fwd(hc, Qd, Kd, Vd, wl.q_begin, sg, ns, O, lse)
    torch.cuda.synchronize()
    assert torch.isfinite(O.float()).all()
    assert torch.equal(O, run.O)


def test_backward_is_deterministic_and_writes_only_active_rows():
    wl = synth.WORKLOADS["qwen3_8b_2k"].with_budget()
    wl = replace(wl, q_begin=1024, n_q=1024, grad_begin=512)
    inp = P.make_inputs(wl, True)
    run = P.gpu_run(wl, inp, True)
    hc = P.hcfg_of(wl)
    Q, K, V, dO = (P.to_dev(x) for x in (inp.Q, inp.K, inp.V, inp.dO))
    sg = torch.from_numpy(run.sel_groups).cuda()
    ns = torch.from_numpy(run.n_sel).cuda()
    n_act = wl.q_begin + wl.n_q - wl.grad_begin
    canary = -12345.0
    dK = torch.full((n_act + 64, wl.n_kv_heads, wl.head_dim), canary, device="cuda")
    dV = torch.full_like(dK, canary)
    dQ = torch.full((wl.n_q + 64, wl.n_q_heads, wl.head_dim), canary, device="cuda")
    ws = torch.empty(hga.workspace_size(hc, hga.OP_BWD, wl.q_begin, wl.n_q, wl.grad_begin), dtype=torch.uint8,
                     device="cuda")
    hga.attend_bwd(hc, Q, K, V, run.O, dO, run.lse, wl.q_begin, wl.grad_begin, sg, ns, dQ, dK, dV,
                   ws, run.o32)
    torch.cuda.synchronize()
    assert torch.equal(dK[:n_act], run.dK) and torch.equal(dV[:n_act], run.dV)
    assert torch.equal(dQ[:wl.n_q], run.dQ)
    assert (dK[n_act:] == canary).all() and (dV[n_act:] == canary).all()
    assert (dQ[wl.n_q:] == canary).all()


# ------------------------------------------------------------------ 131K planted

def test_131k_routing_parity_and_planted_recovery():
    wl = synth.WORKLOADS["qwen3_8b_131k_planted"]
    cfg = P.cfg_of(wl)
    say("[131k] generating inputs")
    inp = P.make_inputs(wl, False)
    say("[131k] GPU route + forward")
    run = P.gpu_run(wl, inp, False)
    say("[131k] oracle summaries + routing")
    cs, gs = orc.summaries(inp.K, cfg)
    _check_summaries(wl, run, cs, gs)
    ro = orc.route(inp.Q, cs, gs, cfg, 0, wl.n_q)
    rep = P.compare_routing(wl, run, ro, gs, inp.Q)
    say(f"[131k] routing exact={rep.exact} near_ties={rep.near_ties} mismatches={rep.mismatches}")
    assert rep.mismatches == 0, rep.detail
    pl = synth.plant(wl)
    planted = set(pl.groups.reshape(-1).tolist())
    for blk in pl.probe_blocks:
        for h in range(wl.n_kv_heads):
            assert list(run.sel_chunks[blk, h]) == list(pl.chunks)
            assert set(run.sel_groups[blk, h, :run.n_sel[blk, h]].tolist()) <= planted
    say("[131k] oracle forward on sampled blocks")
    blocks = sorted(set(range(0, wl.n_q // 64, 64)) | set(int(b) for b in pl.probe_blocks))
    O, lse = orc.attend_fwd(inp.Q, inp.K, inp.V, cfg, 0, wl.n_q, run.sel_groups, run.n_sel,
                            blocks=blocks)
    rows = np.concatenate([np.arange(b * 64, (b + 1) * 64) for b in blocks])
    eo = P.max_abs(run.O[rows], O[rows])
    el = P.max_abs(run.lse[rows], lse[rows])
    say(f"[131k] O max-abs {eo:.3g} LSE {el:.3g} on {len(blocks)} blocks")
    assert eo <= P.TOL["bf16"] and el <= P.LSE_TOL["bf16"]


# ------------------------------------------------------------------ dense baseline

def _dense_run(wl, backward):
    """Dense causal attention through the routed kernels: a sink window
    covering the context and no routed chunks or groups."""
    hc = P.hcfg_of(wl)
    T = wl.q_begin + wl.n_q
    inp = P.make_inputs(wl, backward)
    Q, K, V = P.to_dev(inp.Q), P.to_dev(inp.K), P.to_dev(inp.V)
    n_qb = wl.n_q // 64
    sel = torch.full((n_qb, wl.n_kv_heads, 1), -1, dtype=torch.int32, device="cuda")
    n_sel = torch.zeros(n_qb, wl.n_kv_heads, dtype=torch.int32, device="cuda")
    O = torch.empty_like(Q)
    lse = torch.empty(wl.n_q, wl.n_q_heads, device="cuda")
    o32 = torch.empty(wl.n_q, wl.n_q_heads, wl.head_dim, device="cuda") if backward else None
    hga.attend_fwd(hc, Q, K, V, wl.q_begin, sel, n_sel, O, lse, o32)
    grads = None
    if backward:
        dO = P.to_dev(inp.dO)
        n_act = T - wl.grad_begin
        dQ = torch.empty(wl.n_q, wl.n_q_heads, wl.head_dim, device="cuda")
        dK = torch.empty(n_act, wl.n_kv_heads, wl.head_dim, device="cuda")
        dV = torch.empty_like(dK)
        ws = torch.empty(hga.workspace_size(hc, hga.OP_BWD, wl.q_begin, wl.n_q, wl.grad_begin),
                         dtype=torch.uint8, device="cuda")
        hga.attend_bwd(hc, Q, K, V, O, dO, lse, wl.q_begin, wl.grad_begin, sel, n_sel, dQ, dK, dV, ws, o32)
        grads = (dQ, dK, dV)
    torch.cuda.synchronize()
    return inp, O, lse, grads, sel.cpu().numpy(), n_sel.cpu().numpy()


def test_dense_forward_and_backward_match_the_oracle_at_2k():
    """Dense causal attention, forward and backward, at 2K (one segment,
    every token differentiable), element by element against the oracle run
    with the same configuration (a sink window covering the context, no
    routed chunks: the oracle's routed set is then every earlier token)."""
    wl = replace(synth.WORKLOADS["qwen3_8b_2k"], top_chunks=0, top_groups=0, sink_tokens=2048)
    say("[dense] T=2048 fwd+bwd, oracle")
    inp, O, lse, (dQ, dK, dV), sel, n_sel = _dense_run(wl, True)
    cfg = P.cfg_of(wl)
    assert (orc.routed_tokens(31, np.zeros(0, np.int64), cfg) == np.arange(2048)).all()
    Oo, lo = orc.attend_fwd(inp.Q, inp.K, inp.V, cfg, 0, wl.n_q, sel, n_sel)
    oQ, oK, oV = orc.attend_bwd(inp.Q, inp.K, inp.V, inp.dO, cfg, 0, wl.n_q, 0, sel, n_sel)
    errs = [P.max_abs(O, Oo), P.max_abs(lse, lo), P.max_abs(dQ, oQ), P.max_abs(dK, oK), P.max_abs(dV, oV)]
    say(f"[dense] O {errs[0]:.3g} LSE {errs[1]:.3g} dQ {errs[2]:.3g} dK {errs[3]:.3g} dV {errs[4]:.3g}")
    assert errs[1] <= P.LSE_TOL["bf16"]
    assert max(errs[0], errs[2], errs[3], errs[4]) <= P.TOL["bf16"]


def test_dense_baseline_matches_the_oracle_on_sampled_blocks():
    """The dense forward the HGA forward is measured against, at 4K: every
    row of sampled blocks against the oracle (sink window covering the
    context, no routed chunks)."""
    base = synth.WORKLOADS["qwen3_8b_131k_planted"]
    T = 4096
    wl = replace(base, T=T, n_q=T, top_chunks=0, top_groups=0, sink_tokens=T)
    say(f"[dense] T={T} bf16 Hq=32 Hkv=8 d=128")
    inp, O, lse, _, sel, n_sel = _dense_run(wl, False)
    blocks = [0, 13, 40, T // 64 - 1]
    Oo, lo = orc.attend_fwd(inp.Q, inp.K, inp.V, P.cfg_of(wl), 0, T, sel, n_sel, blocks=blocks)
    rows = np.concatenate([np.arange(b * 64, (b + 1) * 64) for b in blocks])
    eo, el = P.max_abs(O[rows], Oo[rows]), P.max_abs(lse[rows], lo[rows])
    say(f"[dense] O max-abs {eo:.3g} LSE {el:.3g} on {len(blocks)} blocks")
    assert eo <= P.TOL["bf16"] and el <= P.LSE_TOL["bf16"]
