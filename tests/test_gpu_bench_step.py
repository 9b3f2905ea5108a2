"""GPU parity of the benchmarked 16K training step, call for call.

bench.py times one Qwen3-8B layer over 16,384 tokens as sixteen 1,024-token
segments (Sec. 2.2: segment-wise backward, history detached). Each segment
makes three C-ABI calls: hga_build_summaries of the segment's keys,
hga_route_attend_fwd, and hga_attend_bwd with grad_begin at the segment
start; the backwards alternate over two side streams (a workspace each)
beside the next segments' forwards and each other, with their dK/dV work
never split. The benchmark forms the backward's row term from the bf16 O;
the step with the optional float32 copy of O is checked too. This test runs
that very step once (``bench.SegmentedStep.step``, the schedule the
benchmark replays) and then compares every segment's routing, O, LSE, dQ, dK
and dV with the CPU oracle on the same seeded inputs. Segment 0 covers
blocks with no sink window and no candidate chunk inside the fused routing +
forward kernel, and the heaviest unsplit dK/dV items. The same step in one
stream, and the overlapped step again, must give the same bits.
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


@pytest.mark.parametrize("o_f32", [False, True])
def test_benched_16k_step_every_segment_matches_oracle(o_f32):
    import bench

    wl = synth.WORKLOADS["qwen3_8b_16k_seg1k"]
    seg = bench.SEGMENT
    st = bench.SegmentedStep(wl, o_f32=o_f32)
    cfg = P.cfg_of(wl)
    inp = P.Inputs(synth.queries(wl, 0, wl.T), synth.keys(wl, 0, wl.T), synth.values(wl, 0, wl.T),
                   synth.grad_output(wl, 0, wl.T))
    cs, gs = orc.summaries(inp.K, cfg, wl.T)
    tol = P.TOL["bf16"]
    worst = {"O": 0.0, "lse": 0.0, "dQ": 0.0, "dK": 0.0, "dV": 0.0}
    near = 0
    say(f"[bench-step] one step, backwards beside the next forwards (float32 O: {o_f32})")
    st.step()
    torch.cuda.synchronize()
    for s in range(wl.T // seg):
        t0, t1 = s * seg, (s + 1) * seg
        say(f"[bench-step] segment {s}: tokens [{t0}, {t1})")
        ws = replace(wl, T=t1, q_begin=t0, n_q=seg, grad_begin=t0)
        rb = st.rbs[s]
        run = P.GpuRun(st.cs, st.gs, rb.sel_chunks.cpu().numpy(), rb.sel_groups.cpu().numpy(),
                       rb.n_sel_groups.cpu().numpy(), st.O[t0:t1], st.lse[t0:t1])
        q = inp.Q[t0:t1]
        ro = orc.route(q, cs, gs, cfg, t0, seg)
        rep = P.compare_routing(ws, run, ro, gs, q)
        assert rep.mismatches == 0, (s, rep.detail)
        near += rep.near_ties
        sel, n = run.sel_groups, run.n_sel
        O, lse = orc.attend_fwd(q, inp.K, inp.V, cfg, t0, seg, sel, n)
        dQ, dK, dV = orc.attend_bwd(q, inp.K, inp.V, inp.dO[t0:t1], cfg, t0, seg, t0, sel, n)
        errs = {"O": P.max_abs(run.O, O), "lse": P.max_abs(run.lse, lse), "dQ": P.max_abs(st.dQ[t0:t1], dQ),
                "dK": P.max_abs(st.dK[t0:t1], dK), "dV": P.max_abs(st.dV[t0:t1], dV)}
        say(f"[bench-step] segment {s}: routing exact={rep.exact} near_ties={rep.near_ties} "
            + " ".join(f"{k} {v:.3g}" for k, v in errs.items()))
        for k, v in errs.items():
            worst[k] = max(worst[k], v)
        assert errs["lse"] <= P.LSE_TOL["bf16"], (s, errs)
        assert max(errs["O"], errs["dQ"], errs["dK"], errs["dV"]) <= tol, (s, errs)
    # the summary tables the step built segment by segment, bit for bit
    for got, ref in ((st.cs, cs), (st.gs, gs)):
        g = hga.summary_rows(got).cpu().numpy()[:, :ref.shape[1]]
        assert np.array_equal(g.view(np.int32), ref.astype(np.float32).view(np.int32))
    say(f"[bench-step] all 16 segments within the bars; worst {worst}; near-ties {near}")
    # the same step in one stream, and the overlapped step once more, give
    # the same bits (no race between the side streams' workspaces)
    keep = {k: getattr(st, k).clone() for k in ("O", "lse", "dQ", "dK", "dV")}
    for overlap in (False, True):
        for k in keep:
            getattr(st, k).fill_(float("nan"))
        st.overlap = overlap
        st.step()
        torch.cuda.synchronize()
        for k, v in keep.items():
            assert torch.equal(getattr(st, k), v), (overlap, k)
