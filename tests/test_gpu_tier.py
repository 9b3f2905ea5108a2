"""GPU parity of the tiered storage path (Sec. 2.2, Fig. 2; Sec. 2.1 item 2):
history K/V and the full group-summary table in pinned host memory, chunk
summaries and a bounded group-summary cache in device memory, the routed
exact K/V staged into a compact device working set before attention.

The 16K training step runs segment by segment as a trainer would: build the
segment's summaries (group summaries straight into the host table), route
with the cache, update the cache, stage the routed rows (history rows read
from host memory), forward and backward over the working set, then move the
segment's K/V to the host store. Every segment's routing tables, O, LSE, dQ,
dK and dV must equal those of the device-resident path bit for bit (the same
step as the benchmark times, itself compared with the oracle), and the hit
flags must equal the oracle's model of the cache (reading R15).
"""

import sys

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


def _tiered_step(wl, n_slots, segments):
    """Run `segments` segments of `wl` through the tiered path; returns the
    per-segment outputs and the cache hit flags."""
    hc = P.hcfg_of(wl)
    T, seg = wl.T, 1024
    Hkv, d = wl.n_kv_heads, wl.head_dim
    gpc = 64 // wl.group_size
    Kall, Vall = P.to_dev(synth.keys(wl)), P.to_dev(synth.values(wl))
    Qall, dOall = P.to_dev(synth.queries(wl)), P.to_dev(synth.grad_output(wl))
    # host tiers: the detached history and the full group-summary table
    K_host = torch.empty(T, Hkv, d, dtype=torch.bfloat16, pin_memory=True)
    V_host = torch.empty_like(K_host, pin_memory=True)
    g_host = torch.zeros(Hkv, d // 4, T // wl.group_size, 4, pin_memory=True)
    kh, vh, gh = hga.host_view(K_host), hga.host_view(V_host), hga.host_view(g_host)
    hs = hga.Strides(K_host.stride(0), K_host.stride(1))
    group_cap = g_host.shape[2]
    # device: chunk summaries, the cache, the active segment and the working set
    chunk_sum = torch.zeros(Hkv, d // 4, T // 64, 4, device="cuda")
    cache = hga.alloc_group_cache(hc, n_slots, T // 64)
    hga.group_cache_clear(hc, cache)
    rb = hga.alloc_route(hc, 0, seg)
    hit = torch.full((seg // 64, Hkv, max(wl.top_chunks, 1)), -7, dtype=torch.int32, device="cuda")
    r_cap = hga.gathered_rows(hc)
    Kc = torch.empty(seg // 64, Hkv, r_cap, d, dtype=torch.bfloat16, device="cuda")
    Vc = torch.empty_like(Kc)
    K_act = torch.empty(seg, Hkv, d, dtype=torch.bfloat16, device="cuda")
    V_act = torch.empty_like(K_act)
    O = torch.empty(seg, wl.n_q_heads, d, dtype=torch.bfloat16, device="cuda")
    lse = torch.empty(seg, wl.n_q_heads, device="cuda")
    o32 = torch.empty(seg, wl.n_q_heads, d, device="cuda")
    dQ = torch.empty(seg, wl.n_q_heads, d, device="cuda")
    dK = torch.empty(seg, Hkv, d, device="cuda")
    dV = torch.empty_like(dK)
    ws = torch.empty(max(hga.workspace_size(hc, hga.OP_BWD, s * seg, seg, s * seg) for s in range(segments)),
                     dtype=torch.uint8, device="cuda")
    ks = hga.Strides(K_act.stride(0), K_act.stride(1))
    out = []
    for s in range(segments):
        t0, t1 = s * seg, (s + 1) * seg
        K_act.copy_(Kall[t0:t1])
        V_act.copy_(Vall[t0:t1])
        q, do = Qall[t0:t1], dOall[t0:t1]
        hga.build_summaries_raw(hc, hga.shifted_rows(K_act, t0), ks, t0, t1, chunk_sum, gh, group_cap)
        hit.fill_(-7)
        hga.route_cached(hc, q, t0, chunk_sum, gh, group_cap, cache, rb.sel_chunks, rb.sel_groups,
                         rb.n_sel_groups, hit, rb.workspace)
        hga.group_cache_update(hc, cache, gh, group_cap, t0, seg, rb.sel_chunks, hit)
        hga.gather_tiered(hc, kh, vh, hs, t0, K_act, V_act, t0, seg, rb.sel_groups, rb.n_sel_groups, Kc, Vc)
        hga.attend_gathered_fwd(hc, q, Kc, Vc, t0, rb.n_sel_groups, O, lse, o32)
        hga.attend_gathered_bwd(hc, q, Kc, Vc, K_act, V_act, t0, O, do, lse, t0, t0, rb.sel_groups,
                                rb.n_sel_groups, dQ, dK, dV, ws, o32)
        # the segment becomes history: its K/V move to the host store
        K_host[t0:t1].copy_(K_act, non_blocking=True)
        V_host[t0:t1].copy_(V_act, non_blocking=True)
        torch.cuda.synchronize()
        out.append({k: v.clone() for k, v in (("sel_chunks", rb.sel_chunks), ("sel_groups", rb.sel_groups),
                                              ("n_sel", rb.n_sel_groups), ("O", O), ("lse", lse), ("dQ", dQ),
                                              ("dK", dK), ("dV", dV), ("hit", hit))})
    return out


@pytest.mark.parametrize("n_slots", [32, 4096])
def test_tiered_step_equals_resident_step_and_cache_model(n_slots):
    import bench

    wl = synth.WORKLOADS["qwen3_8b_16k_seg1k"]
    segments = wl.T // 1024
    say(f"[tier] 16K step, {segments} segments, {n_slots} cache slots per kv head")
    tiered = _tiered_step(wl, n_slots, segments)
    st = bench.SegmentedStep(wl)
    calls = []
    for s in range(segments):
        t0, t1 = s * 1024, (s + 1) * 1024
        for _, fn in st.calls(s):
            fn()
        torch.cuda.synchronize()
        tr, rb = tiered[s], st.rbs[s]
        assert torch.equal(tr["sel_chunks"], rb.sel_chunks), s
        assert torch.equal(tr["sel_groups"], rb.sel_groups), s
        assert torch.equal(tr["n_sel"], rb.n_sel_groups), s
        assert torch.equal(tr["O"], st.O[t0:t1]), s
        assert torch.equal(tr["lse"], st.lse[t0:t1]), s
        for k, ref in (("dQ", st.dQ[t0:t1]), ("dK", st.dK[t0:t1]), ("dV", st.dV[t0:t1])):
            assert torch.equal(tr[k], ref), (s, k)
        calls.append(tr["sel_chunks"].cpu().numpy())
    want = orc.group_cache_hits(calls, wl.n_kv_heads, n_slots)
    n_hit = n_req = 0
    for s in range(segments):
        got = tiered[s]["hit"].cpu().numpy()
        chosen = calls[s] >= 0
        np.testing.assert_array_equal(got[chosen], want[s][chosen])
        n_hit += int((want[s] == 1).sum())
        n_req += int(chosen.sum())
    say(f"[tier] equal to the resident step; cache hits {n_hit}/{n_req} = {n_hit / max(n_req, 1):.3f}")


def test_gathered_backward_matches_the_oracle():
    """The backward over compact rows on its own, 32K sweep segment: dQ from
    the working set, dK/dV from the active rows; against the oracle."""
    wl = synth.WORKLOADS["qwen3_8b_32k_sweep"].with_budget(group_size=8, top_chunks=8, top_groups=32)
    inp = P.make_inputs(wl, True)
    run = P.gpu_run(wl, inp, True)
    hc, cfg = P.hcfg_of(wl), P.cfg_of(wl)
    t0, n = wl.q_begin, wl.n_q
    Q, K, V, dO = (P.to_dev(x) for x in (inp.Q, inp.K, inp.V, inp.dO))
    sg = torch.from_numpy(run.sel_groups).cuda()
    ns = torch.from_numpy(run.n_sel).cuda()
    Kc = torch.empty(n // 64, wl.n_kv_heads, hga.gathered_rows(hc), wl.head_dim, dtype=torch.bfloat16,
                     device="cuda")
    Vc = torch.empty_like(Kc)
    hga.gather_routed(hc, K, V, t0, n, sg, ns, Kc, Vc)
    dQ, dK, dV = torch.empty_like(run.dQ), torch.empty_like(run.dK), torch.empty_like(run.dV)
    ws = torch.empty(hga.workspace_size(hc, hga.OP_BWD, t0, n, wl.grad_begin), dtype=torch.uint8, device="cuda")
    K_act, V_act = K[wl.grad_begin:].contiguous(), V[wl.grad_begin:].contiguous()
    hga.attend_gathered_bwd(hc, Q, Kc, Vc, K_act, V_act, wl.grad_begin, run.O, dO, run.lse, t0, wl.grad_begin,
                            sg, ns, dQ, dK, dV, ws, run.o32)
    torch.cuda.synchronize()
    assert torch.equal(dQ, run.dQ) and torch.equal(dK, run.dK) and torch.equal(dV, run.dV)
    oQ, oK, oV = orc.attend_bwd(inp.Q, inp.K, inp.V, inp.dO, cfg, t0, n, wl.grad_begin, run.sel_groups, run.n_sel)
    errs = (P.max_abs(dQ, oQ), P.max_abs(dK, oK), P.max_abs(dV, oV))
    say(f"[tier] gathered backward dQ {errs[0]:.3g} dK {errs[1]:.3g} dV {errs[2]:.3g}")
    assert max(errs) <= P.TOL["bf16"]
