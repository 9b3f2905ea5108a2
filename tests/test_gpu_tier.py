"""GPU parity of the tiered storage path (Sec. 2.2, Fig. 2; Sec. 2.1 item 2):
history K/V and the full group-summary table in pinned host memory, chunk
summaries and a bounded group-summary cache in device memory, the routed
exact K/V staged into a compact device working set before attention.

The 16K training step runs as the benchmark times it (``bench.TieredStep``):
per segment, build the summaries (group summaries straight into the host
table), route with the cache, update the cache, stage the routed rows,
forward and backward over the working set. The device keeps the last two
segments' K/V; an older segment moves to the host store on a copy stream
beside the next segments' work, and the staging of a later segment waits for
it. Every segment's routing tables, O, LSE, dQ, dK and dV must equal those of
the device-resident path bit for bit (the same step as the benchmark times,
itself compared with the oracle), and the hit flags must equal the oracle's
model of the cache (reading R15).
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


@pytest.mark.parametrize("n_slots", [32, 4096])
def test_tiered_step_equals_resident_step_and_cache_model(n_slots):
    import bench

    wl = synth.WORKLOADS["qwen3_8b_16k_seg1k"]
    segments = wl.T // 1024
    say(f"[tier] 16K step, {segments} segments, {n_slots} cache slots per kv head")
    ts = bench.TieredStep(wl, n_slots)
    for s in range(segments):
        ts.hits[s].fill_(-7)
    ts.step()
    torch.cuda.synchronize()
    tiered = [{"sel_chunks": ts.rbs[s].sel_chunks, "sel_groups": ts.rbs[s].sel_groups,
               "n_sel": ts.rbs[s].n_sel_groups, "hit": ts.hits[s],
               "O": ts.O[s * 1024:(s + 1) * 1024], "lse": ts.lse[s * 1024:(s + 1) * 1024],
               "dQ": ts.dQ[s * 1024:(s + 1) * 1024], "dK": ts.dK[s * 1024:(s + 1) * 1024],
               "dV": ts.dV[s * 1024:(s + 1) * 1024]} for s in range(segments)]
    # the host store holds every detached segment's keys and values
    n_det = segments - ts.dev_segs
    assert torch.equal(ts.K_host[:n_det * 1024], ts.Kall[:n_det * 1024].cpu())
    assert torch.equal(ts.V_host[:n_det * 1024], ts.Vall[:n_det * 1024].cpu())
    st = bench.SegmentedStep(wl)
    st.overlap = False
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
    # a second step (the cache cleared again at its start) gives the same bits
    keep = [{k: v.clone() for k, v in tr.items()} for tr in tiered]
    ts.step()
    torch.cuda.synchronize()
    for s in range(segments):
        for k, v in keep[s].items():
            assert torch.equal(tiered[s][k], v), (s, k)


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
