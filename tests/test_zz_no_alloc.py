"""hga_attend_bwd_noalloc against hga_attend_bwd, through the C ABI.

The entry point that allocates nothing takes the backward's workspace from
the library's static per-device buffer. Two calls in a row, the second on a
smaller input, must give bit for bit the results of the workspace entry point
(the backward is deterministic), and a call that needs more scratch than the
buffer holds must be rejected before anything is launched.
"""

import sys
from dataclasses import replace

import pytest
import torch

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


def _noalloc_matches(wl):
    hc = P.hcfg_of(wl)
    need = hga.workspace_size(hc, hga.OP_BWD, wl.q_begin, wl.n_q, wl.grad_begin)
    say(f"[noalloc] q_begin={wl.q_begin} n_q={wl.n_q} grad_begin={wl.grad_begin} scratch {need} B")
    assert 0 < need <= hga.NOALLOC_SCRATCH_BYTES
    inp = P.make_inputs(wl, True)
    run = P.gpu_run(wl, inp, True)  # summaries, route, fwd, bwd with a caller workspace
    Q, K, V, dO = (P.to_dev(x) for x in (inp.Q, inp.K, inp.V, inp.dO))
    sg = torch.from_numpy(run.sel_groups).cuda()
    ns = torch.from_numpy(run.n_sel).cuda()
    dQ, dK, dV = torch.full_like(run.dQ, 7.0), torch.full_like(run.dK, 7.0), torch.full_like(run.dV, 7.0)
    hga.attend_bwd_noalloc(hc, Q, K, V, run.O, dO, run.lse, wl.q_begin, wl.grad_begin, sg, ns, dQ, dK, dV,
                           run.o32)
    torch.cuda.synchronize()
    assert torch.equal(dQ, run.dQ) and torch.equal(dK, run.dK) and torch.equal(dV, run.dV)


def test_noalloc_backward_equals_workspace_backward_twice_then_smaller():
    base = synth.WORKLOADS["qwen3_8b_2k"]
    # 2,048 queries from token 0: D plus the split dK/dV partials (~34 MB)
    _noalloc_matches(base)
    # then a smaller call on the same buffer: 1,024 queries, dK/dV from 1,024
    _noalloc_matches(replace(base, q_begin=1024, n_q=1024, grad_begin=1024))


def test_noalloc_rejects_calls_beyond_its_scratch():
    hc = P.hcfg_of(synth.WORKLOADS["qwen3_8b_2k"])
    assert hga.workspace_size(hc, hga.OP_BWD, 0, 4096, 0) > hga.NOALLOC_SCRATCH_BYTES
    x = torch.zeros(4096, 32, 128, dtype=torch.bfloat16, device="cuda")
    kv = torch.zeros(4096, 8, 128, dtype=torch.bfloat16, device="cuda")
    f = torch.zeros(4096, 32, 128, device="cuda")
    fk = torch.zeros(4096, 8, 128, device="cuda")
    lse = torch.zeros(4096, 32, device="cuda")
    sg = torch.zeros(64, 8, 16, dtype=torch.int32, device="cuda")
    ns = torch.zeros(64, 8, dtype=torch.int32, device="cuda")
    with pytest.raises(hga.HgaError) as e:
        hga.attend_bwd_noalloc(hc, x, kv, kv, x, x, lse, 0, 0, sg, ns, f, fk, fk)
    assert e.value.status == -3
