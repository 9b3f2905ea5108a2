"""GPU parity of the stand-alone gather (hga_gather_routed) and of the
forward over its compact rows (hga_attend_gathered_fwd), both through the C
ABI. Routing comes from the oracle, so every expected value is the oracle's:

* the gather is index work, so its rows must equal the oracle's routed token
  rows bit for bit, in the tile order [sink | local | selected groups], with
  zero rows up to the next 64 and untouched rows after;
* the forward over compact rows must give bit for bit what hga_attend_fwd
  gives on the same routing (same tiles, same arithmetic), and match the
  oracle's attention within the bf16 / fp32 bars.
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


BASE = synth.Workload("gather", T=2048, n_q_heads=8, n_kv_heads=2, head_dim=128, dtype="bf16",
                      seed=31, q_begin=1024, n_q=1024, grad_begin=1024, key_offset="normal",
                      backward=False)
CASES = {
    "default": BASE,
    "ragged": replace(BASE, top_groups=13),                       # partial last tile
    "no_sink": replace(BASE, sink_tokens=0, local_tokens=64),
    "g16_d64": replace(BASE, group_size=16, top_groups=9, head_dim=64, q_begin=0, n_q=2048),
    "fp32": replace(synth.WORKLOADS["tiny_fp32_1k"], backward=False),
}


def _setup(wl):
    cfg = P.cfg_of(wl)
    inp = P.make_inputs(wl, False)
    cs, gs = orc.summaries(inp.K, cfg, wl.q_begin + wl.n_q)
    ro = orc.route(inp.Q, cs, gs, cfg, wl.q_begin, wl.n_q)
    sel = ro.sel_groups if wl.top_groups else np.full((wl.n_q // 64, wl.n_kv_heads, 1), -1, np.int32)
    return cfg, inp, ro, torch.from_numpy(np.ascontiguousarray(sel)).cuda(), \
        torch.from_numpy(ro.n_sel_groups).cuda()


def _tile_order_tokens(abs_block, groups, cfg):
    sink_end, local_start, block_end = orc.windows(abs_block, cfg)
    g = cfg.group_size
    parts = [np.arange(0, sink_end), np.arange(local_start, block_end)]
    parts += [np.arange(j * g, (j + 1) * g) for j in sorted(groups)]
    return np.concatenate(parts).astype(np.int64)


@pytest.mark.parametrize("name", list(CASES))
def test_gather_routed_rows_bit_exact(name):
    wl = CASES[name]
    say(f"[gather] {name}: T={wl.q_begin + wl.n_q} q_begin={wl.q_begin} g={wl.group_size} "
        f"kg={wl.top_groups} d={wl.head_dim} {wl.dtype}")
    cfg, inp, ro, sel, ns = _setup(wl)
    hc = P.hcfg_of(wl)
    r_cap = hga.gathered_rows(hc) + 64  # one spare tile per slot must stay untouched
    K, V = P.to_dev(inp.K), P.to_dev(inp.V)
    shape = (wl.n_q // 64, wl.n_kv_heads, r_cap, wl.head_dim)
    sentinel = 0x7FC1 if wl.dtype == "bf16" else 0x7FC00001
    if wl.dtype == "bf16":
        Kc = torch.full(shape, sentinel, dtype=torch.int16, device="cuda").view(torch.bfloat16)
    else:
        Kc = torch.full(shape, sentinel, dtype=torch.int32, device="cuda").view(torch.float32)
    Vc = Kc.clone()
    hga.gather_routed(hc, K, V, wl.q_begin, wl.n_q, sel, ns, Kc, Vc)
    torch.cuda.synchronize()
    kc, vc = P.to_np(Kc), P.to_np(Vc)
    bits = (lambda x: x) if wl.dtype == "bf16" else (lambda x: np.ascontiguousarray(x).view(np.int32))
    kc, vc = bits(kc), bits(vc)
    Kr, Vr = bits(inp.K), bits(inp.V)
    for b in range(wl.n_q // 64):
        for h in range(wl.n_kv_heads):
            toks = _tile_order_tokens(wl.q_begin // 64 + b, ro.sel_groups[b, h, :ro.n_sel_groups[b, h]], cfg)
            R = len(toks)
            assert sorted(toks.tolist()) == sorted(orc.routed_tokens(
                wl.q_begin // 64 + b, ro.sel_groups[b, h, :ro.n_sel_groups[b, h]], cfg).tolist())
            pad = -(-R // 64) * 64
            np.testing.assert_array_equal(kc[b, h, :R], Kr[toks, h])
            np.testing.assert_array_equal(vc[b, h, :R], Vr[toks, h])
            assert (kc[b, h, R:pad] == 0).all() and (vc[b, h, R:pad] == 0).all()
            assert (kc[b, h, pad:] == np.array(sentinel).astype(kc.dtype)).all()
            assert (vc[b, h, pad:] == np.array(sentinel).astype(vc.dtype)).all()


@pytest.mark.parametrize("name", list(CASES))
def test_attend_gathered_equals_attend_fwd(name):
    wl = CASES[name]
    say(f"[gathered fwd] {name}")
    cfg, inp, ro, sel, ns = _setup(wl)
    hc = P.hcfg_of(wl)
    Q, K, V = P.to_dev(inp.Q), P.to_dev(inp.K), P.to_dev(inp.V)
    r_cap = hga.gathered_rows(hc)
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    Kc = torch.empty(wl.n_q // 64, wl.n_kv_heads, r_cap, wl.head_dim, dtype=dt, device="cuda")
    Vc = torch.empty_like(Kc)
    outs = []
    for gathered in (False, True):
        O = torch.empty_like(Q)
        lse = torch.empty(wl.n_q, wl.n_q_heads, device="cuda")
        o32 = torch.empty(wl.n_q, wl.n_q_heads, wl.head_dim, device="cuda")
        if gathered:
            hga.gather_routed(hc, K, V, wl.q_begin, wl.n_q, sel, ns, Kc, Vc)
            hga.attend_gathered_fwd(hc, Q, Kc, Vc, wl.q_begin, ns, O, lse, o32)
        else:
            hga.attend_fwd(hc, Q, K, V, wl.q_begin, sel, ns, O, lse, o32)
        torch.cuda.synchronize()
        outs.append((O, lse, o32))
    for x, y in zip(*outs):
        assert torch.equal(x, y)
    Oref, lref = orc.attend_fwd(inp.Q, inp.K, inp.V, cfg, wl.q_begin, wl.n_q, ro.sel_groups,
                                ro.n_sel_groups)
    eo, el = P.max_abs(outs[1][0], Oref), P.max_abs(outs[1][1], lref)
    say(f"[gathered fwd] O max-abs {eo:.3g} LSE {el:.3g}")
    assert eo <= P.TOL[wl.dtype] and el <= P.LSE_TOL[wl.dtype]
