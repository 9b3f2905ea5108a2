#!/usr/bin/env python3
"""Benchmark of the HGA route + attend hot path on one MI355X.

Headline step (all steps of the path, forward and backward): one Qwen3-8B
attention layer (32 query heads, 8 kv heads, head dim 128, bf16) over 16,384
tokens processed as sixteen 1,024-token segments. Per segment: key summaries
of the new tokens, two-level routing of the segment's query blocks, routed
attention forward (with the float32 O the backward uses) and backward with
dK/dV for the segment's own tokens only; history K/V stays resident in HBM.
Budget: 64-token chunks, 8-token groups, top 8 chunks then top 16 groups,
sink 64, local 128.

`value` = query tokens per second of that step (16,384 / step time), timed
over replays of a HIP graph of the step (inputs already resident in HBM).
Per-call durations come from HIP events around each call in an eager pass
over the same step, launched behind a short GPU spin so that the host never
starves the queue; they give the phase split and the roofline of the
dominant kernel. Also reported: the same layer's forward over 131,072 tokens
(top 16 chunks / 32 groups, local 256) and the same budget at 16K, 32K and
64K (per-token cost against context length), the 32K routing sweep with
scoring and attention timed separately, and the CPU oracle on a bounded
sample.
"""

from __future__ import annotations

import argparse
import ctypes
import dataclasses
import json
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2607_15105_amd import hga, synth  # noqa: E402

METRIC = "routed-attention query tokens/s per layer (fwd, fwd+bwd) at 16K/131K; HBM GB/s"
HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
SEGMENT = 1024
# Side streams of the overlapped step's backwards (even and odd segments):
# consecutive backwards run beside each other, so one's last workgroups do
# not leave the chip idle before the next starts (three measured no better).
N_SIDE = 2


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def to_dev(x: np.ndarray) -> torch.Tensor:
    if x.dtype == np.uint16:
        return torch.from_numpy(x.view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(x).cuda()


def hcfg(wl: synth.Workload) -> hga.Config:
    return hga.make_config(wl.n_q_heads, wl.n_kv_heads, wl.head_dim, group_size=wl.group_size,
                           top_chunks=wl.top_chunks, top_groups=wl.top_groups,
                           sink_tokens=wl.sink_tokens, local_tokens=wl.local_tokens)


# The segmented step's backwards overlap each other (two side streams), so
# each takes the least total work: one dK/dV item per (chunk, kv head), never
# split over query-head subsets (a split shortens one call on its own but adds
# list builds and a combine kernel).
STEP_BWD_KV_PARTS = 1


def step_hcfg(wl: synth.Workload) -> hga.Config:
    hc = hcfg(wl)
    hc.bwd_kv_parts = STEP_BWD_KV_PARTS
    return hc


# ----------------------------------------------------------------------------
# Algorithmic work of one call (what the method must touch, not what a kernel
# happens to re-read): flops of the attention products over the visible
# (query, key) pairs, and HBM bytes of inputs read once and outputs written.
# ----------------------------------------------------------------------------

def routed_sizes(wl: synth.Workload, q_begin: int, n_q: int, n_sel: np.ndarray) -> np.ndarray:
    """R[b, h]: routed keys of each (query block, kv head)."""
    b = q_begin // 64 + np.arange(n_q // 64)
    end = (b + 1) * 64
    ls = np.maximum(0, end - wl.local_tokens)
    sink = np.minimum(wl.sink_tokens, ls)
    return (sink + (end - ls))[:, None] + n_sel * wl.group_size


def visible_pairs(wl, q_begin, n_q, n_sel) -> np.ndarray:
    """(query, key) pairs each (query block, kv head) attends: R - 64 keys
    before the block for all 64 rows, plus the causal half of the diagonal
    block."""
    R = routed_sizes(wl, q_begin, n_q, n_sel)
    return 64 * (R - 64) + 64 * 65 // 2


def causal_pairs(q_begin, n_q) -> int:
    """(query, key) pairs of dense causal attention over the call's rows."""
    i = np.arange(q_begin, q_begin + n_q, dtype=np.int64)
    return int((i + 1).sum())


def selection_density(wl, q_begin, n_q, n_sel) -> float:
    """Attended over causal (query, key) pairs, all kv heads: the statistic
    of the paper's Tables 1, 4, 5 and 7."""
    return float(visible_pairs(wl, q_begin, n_q, n_sel).sum()) / (causal_pairs(q_begin, n_q) * wl.n_kv_heads)


def attn_work(wl, q_begin, n_q, n_sel, backward: bool, o_f32: bool = False):
    """(flops, algorithmic bytes, implementation bytes) of one attention call.

    Algorithmic bytes are what the method must move: the routed K/V working
    set of every (block, kv head), Q and O (and dO) at the input dtype, the
    LSE and, for the backward, dQ, dK and dV (float32 outputs). With o_f32
    the forward also writes a float32 copy of O and the backward reads it in
    place of O for the row term D (an optional precision choice, 4 B per
    element): those bytes are returned apart as implementation bytes."""
    R = routed_sizes(wl, q_begin, n_q, n_sel)
    G, d = wl.n_q_heads // wl.n_kv_heads, wl.head_dim
    pairs = visible_pairs(wl, q_begin, n_q, n_sel) * G   # visible pairs per (block, kv head)
    kv_ws = float(R.sum()) * d * 2 * 2                   # K and V rows gathered per (block, head)
    rows = n_q * wl.n_q_heads * d
    o32 = rows * 4 if o_f32 else 0
    if not backward:   # Q in, O out (bf16), LSE out
        return 4.0 * d * pairs.sum(), kv_ws + rows * (2 + 2) + n_q * wl.n_q_heads * 4, o32
    n_act = q_begin + n_q - wl.grad_begin
    # Q, O, dO, LSE in; dQ, dK, dV out (float32)
    return (10.0 * d * pairs.sum(),
            kv_ws + rows * (2 + 2 + 2 + 4) + n_q * wl.n_q_heads * 4 +
            2 * n_act * wl.n_kv_heads * d * 4, o32)


def route_work(wl, q_begin, n_q):
    d = wl.head_dim
    n_qb = n_q // 64
    end = q_begin + n_q
    n_chunks = max(0, (end - wl.local_tokens) // 64 - wl.sink_tokens // 64)
    g_rows = n_qb * wl.n_kv_heads * wl.top_chunks * (64 // wl.group_size)
    qbytes = n_q * wl.n_q_heads * d * 2
    # Q once, the chunk table of the call once, the groups of the chosen chunks per block
    return qbytes + n_chunks * wl.n_kv_heads * d * 4 + g_rows * d * 4


def summary_work(wl, t0, t1):
    return (t1 - t0) * wl.n_kv_heads * wl.head_dim * 2 + \
        ((t1 - t0) // 64 + (t1 - t0) // wl.group_size) * wl.n_kv_heads * wl.head_dim * 4


# ----------------------------------------------------------------------------
# The 16K segmented training step
# ----------------------------------------------------------------------------

def unsplit_bwd_segments(hc):
    """Segments of the 16K step whose backward workspace is D alone (n_q x Hq
    floats rounded up to 256 bytes): no split dK/dV work."""
    dvec = -(-SEGMENT * hc.n_q_heads * 4 // 256) * 256
    return [s for s in range(16)
            if hga.workspace_size(hc, hga.OP_BWD, s * SEGMENT, SEGMENT, s * SEGMENT) == dvec]


_HIP = None


def _hip():
    """The HIP runtime, for the event calls of a launch loop."""
    global _HIP
    if _HIP is None:
        h = ctypes.CDLL("libamdhip64.so")
        h.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        h.hipEventRecord.restype = ctypes.c_int
        h.hipStreamWaitEvent.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_uint]
        h.hipStreamWaitEvent.restype = ctypes.c_int
        h.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
        h.hipEventCreateWithFlags.restype = ctypes.c_int
        h.hipEventDestroy.argtypes = [ctypes.c_void_p]
        h.hipEventDestroy.restype = ctypes.c_int
        _HIP = h
    return _HIP


EVENT_FLAGS = 0x2  # hipEventDisableTiming


def _hip_events(n: int) -> list:
    """n HIP events without timing (a stream waits on one at half the host
    cost of a torch event)."""
    evs = []
    for _ in range(n):
        e = ctypes.c_void_p()
        if _hip().hipEventCreateWithFlags(ctypes.byref(e), EVENT_FLAGS):
            raise RuntimeError("hipEventCreateWithFlags failed")
        evs.append(e)
    return evs


class SegmentedStep:
    """The 16K training step: 16 segments x (summaries, routing + forward,
    backward). Every segment has its own routing tables and output rows, so
    the only orders between calls are their data dependencies: a segment's
    forward needs its own summaries and those of earlier segments (one
    stream), its backward needs its forward. The forward of segment s + 1
    needs nothing from the backward of segment s (gradients do not cross
    segments and nothing updates the inputs within the step), and no
    backward needs another, so with `overlap` the backwards run on two side
    streams (even and odd segments, a workspace each), each after its own
    forward, beside the next segments' forwards and beside each other."""

    def __init__(self, wl: synth.Workload, overlap: bool = True, o_f32: bool = False):
        self.wl = wl
        self.overlap = overlap
        T = wl.T
        n_seg = T // SEGMENT
        self.hc = step_hcfg(wl)
        log(f"[bench] generating {T}-token inputs")
        self.Q = to_dev(synth.queries(wl, 0, T))
        self.K = to_dev(synth.keys(wl, 0, T))
        self.V = to_dev(synth.values(wl, 0, T))
        self.dO = to_dev(synth.grad_output(wl, 0, T))
        self.cs, self.gs = hga.alloc_summaries(self.hc, T)
        self.rbs = [hga.alloc_route(self.hc, s * SEGMENT, SEGMENT) for s in range(n_seg)]
        self.O = torch.empty_like(self.Q)
        self.lse = torch.empty(T, wl.n_q_heads, device="cuda")
        # The row term D = rowsum(dO * O) is formed from the bf16 O, as flash
        # attention's backward forms it; with o_f32 the forward also writes a
        # float32 copy of O (its P not rounded) and D comes from that copy.
        self.o32 = torch.empty(T, wl.n_q_heads, wl.head_dim, device="cuda") if o_f32 else None
        self.dQ = torch.empty(T, wl.n_q_heads, wl.head_dim, device="cuda")
        self.dK = torch.empty(T, wl.n_kv_heads, wl.head_dim, device="cuda")
        self.dV = torch.empty_like(self.dK)
        ws_bytes = max(hga.workspace_size(self.hc, hga.OP_BWD, s, SEGMENT, s) for s in range(0, T, SEGMENT))
        self.bws = [torch.empty(ws_bytes, dtype=torch.uint8, device="cuda") for _ in range(N_SIDE)]
        self.sides = [torch.cuda.Stream() for _ in range(N_SIDE)]
        self.ev_fwd = _hip_events(n_seg)
        self._prep = {}  # prepared calls per (stream, overlap)
        self.n_sel = {}
        self.routing = {}

    def calls(self, s: int):
        """The three ABI calls of segment s, as closures: summaries of its keys,
        routing + forward (one launch at this size), backward."""
        t0, t1 = s * SEGMENT, (s + 1) * SEGMENT
        hc, rb = self.hc, self.rbs[s]
        q, o, lse, do = self.Q[t0:t1], self.O[t0:t1], self.lse[t0:t1], self.dO[t0:t1]
        o32 = self.o32[t0:t1] if self.o32 is not None else None
        dq, dk, dv = self.dQ[t0:t1], self.dK[t0:t1], self.dV[t0:t1]
        return [
            ("summaries", lambda: hga.build_summaries(hc, self.K, t0, t1, self.cs, self.gs)),
            ("route_attend_fwd", lambda: hga.route_attend_fwd(hc, q, self.K, self.V, t0, self.cs, self.gs,
                                                              rb.sel_chunks, rb.sel_groups, rb.n_sel_groups,
                                                              o, lse, rb.workspace, o32)),
            ("attend_bwd", lambda: hga.attend_bwd(hc, q, self.K, self.V, o, do, lse, t0, t0,
                                                  rb.sel_groups, rb.n_sel_groups, dq, dk, dv, self.bws[s % N_SIDE],
                                                  o32)),
        ]

    def __del__(self):
        try:
            for e in self.ev_fwd:
                _hip().hipEventDestroy(e)
        except Exception:  # interpreter shutdown
            pass

    def prepared(self, main):
        """Every segment's ABI calls recorded once with their arguments
        marshalled (hga.record): the summaries and the routing + forward on
        `main`, the backward on `main` too without overlap, else on the side
        stream of its segment's parity. Issuing them then costs one foreign
        call each, so the host stays ahead of the GPU."""
        key = (main.cuda_stream, self.overlap)
        if key not in self._prep:
            calls = []
            for s in range(self.wl.T // SEGMENT):
                c = dict(self.calls(s))
                with hga.record() as fw:
                    c["summaries"]()
                    c["route_attend_fwd"]()
                with torch.cuda.stream(self.sides[s % N_SIDE] if self.overlap else main), hga.record() as bw:
                    c["attend_bwd"]()
                calls.append((fw, bw))
            self._prep[key] = calls
        return self._prep[key]

    def step(self):
        main = torch.cuda.current_stream()
        calls = self.prepared(main)
        if not self.overlap:
            for fw, bw in calls:
                for fn in fw + bw:
                    fn()
            return
        for side in self.sides:  # the backwards start after whatever precedes the step
            side.wait_stream(main)
        hip, ms = _hip(), ctypes.c_void_p(main.cuda_stream)
        ss = [ctypes.c_void_p(side.cuda_stream) for side in self.sides]
        def fwd(s):
            for fn in calls[s][0]:
                fn()
            if hip.hipEventRecord(self.ev_fwd[s], ms):
                raise RuntimeError("hipEventRecord failed")

        def bwd(s):  # after its forward
            if hip.hipStreamWaitEvent(ss[s % N_SIDE], self.ev_fwd[s], 0):
                raise RuntimeError("hipStreamWaitEvent failed")
            for fn in calls[s][1]:
                fn()

        # A stream wait costs the host tens of microseconds. Segment 0's
        # backward is issued at once (the side streams have nothing else to
        # do); every later one after the next segment's forward calls, so
        # that the wait never holds back a forward.
        n = len(calls)
        fwd(0)
        bwd(0)
        for s in range(1, n):
            fwd(s)
            if s >= 2:
                bwd(s - 1)
        if n > 1:
            bwd(n - 1)
        for side in self.sides:  # the step ends with the last backwards
            main.wait_stream(side)


    def record_routing(self):
        """Routing counts of every segment (for the algorithmic work), eagerly."""
        for s in range(self.wl.T // SEGMENT):
            for name, fn in self.calls(s):
                fn()
                if name == "route_attend_fwd":
                    rb = self.rbs[s]
                    self.n_sel[s] = rb.n_sel_groups.cpu().numpy().copy()
                    self.routing[s] = (rb.sel_chunks.cpu().numpy().copy(),
                                       rb.sel_groups.cpu().numpy().copy(), self.n_sel[s])
        torch.cuda.synchronize()

    def density(self, segments=None) -> float:
        """Selection density of the step (or of the given segments): attended
        over causal (query, key) pairs, all kv heads."""
        segs = range(self.wl.T // SEGMENT) if segments is None else segments
        att = sum(float(visible_pairs(self.wl, s * SEGMENT, SEGMENT, self.n_sel[s]).sum()) for s in segs)
        cau = sum(causal_pairs(s * SEGMENT, SEGMENT) * self.wl.n_kv_heads for s in segs)
        return att / cau

    def work(self):
        """Algorithmic (flops, bytes) per call name summed over the step, and
        the backward's per segment."""
        wl, out, bwd = self.wl, {}, []
        for s in range(wl.T // SEGMENT):
            t0 = s * SEGMENT
            wl_s = dataclasses.replace(wl, grad_begin=t0)
            f32 = self.o32 is not None
            f = attn_work(wl_s, t0, SEGMENT, self.n_sel[s], False, f32)
            b = attn_work(wl_s, t0, SEGMENT, self.n_sel[s], True, f32)
            bwd.append(b)
            for k, (fl, by, im) in (("route_attend_fwd", (f[0], f[1] + route_work(wl, t0, SEGMENT), f[2])),
                                    ("attend_bwd", b),
                                    ("summaries", (0.0, summary_work(wl, t0, t0 + SEGMENT), 0.0))):
                a = out.setdefault(k, [0.0, 0.0, 0.0])
                a[0] += fl
                a[1] += by
                a[2] += im
        return out, bwd

    def single_kernel_bwd_segments(self):
        """Segments whose dK/dV work is not split over query-head subsets (the
        backward workspace holds only D), so no combine kernel runs."""
        return unsplit_bwd_segments(self.hc)


_SPIN_CYCLES_PER_MS = None


def _spin_cycles(ms: float) -> int:
    """GPU spin length (torch.cuda._sleep cycles) lasting about `ms`, calibrated once."""
    global _SPIN_CYCLES_PER_MS
    if _SPIN_CYCLES_PER_MS is None:
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        torch.cuda._sleep(1_000_000)
        e1.record()
        torch.cuda.synchronize()
        _SPIN_CYCLES_PER_MS = 1_000_000 / max(e0.elapsed_time(e1), 1e-3)
    return int(_SPIN_CYCLES_PER_MS * ms)


def timed_events(fns_by_name, reps: int, warm: int = 3):
    """Median GPU duration of each named call over `reps` eager passes that
    follow `warm` untimed ones (the paper's timing protocol is the median of
    ten runs after three warm-ups), from HIP events on the launching stream.
    A GPU spin queued ahead of each pass keeps the host ahead of the device,
    so no launch gap lands inside a bracket."""
    samples = {}
    for _ in range(max(warm, 1)):
        t = time.perf_counter()
        for _, fn in fns_by_name():
            fn()
        torch.cuda.synchronize()
        host_ms = (time.perf_counter() - t) * 1e3
    for _ in range(reps):
        pairs = []
        torch.cuda._sleep(_spin_cycles(3.0 * host_ms + 1.0))
        for name, fn in fns_by_name():
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            pairs.append((name, e0, e1))
        torch.cuda.synchronize()
        for name, e0, e1 in pairs:
            samples.setdefault(name, []).append(e0.elapsed_time(e1))
    return {k: float(np.median(v)) for k, v in samples.items()}, {k: len(v) for k, v in samples.items()}


def eager_median_ms(fn, reps: int = 10, warm: int = 3) -> float:
    """Median duration of one eager call of `fn` (which may use several
    streams and ends on the current one) over `reps` runs timed one by one
    with HIP events on the current stream, after `warm` untimed runs. A GPU
    spin queued ahead of each run keeps the host's launches ahead of the
    device."""
    for _ in range(warm):
        t = time.perf_counter()
        fn()
        torch.cuda.synchronize()
        host_ms = (time.perf_counter() - t) * 1e3
    ts = []
    for _ in range(reps):
        torch.cuda._sleep(_spin_cycles(2.0 * host_ms + 1.0))
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        fn()
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1))
    return float(np.median(ts))


def replay_median_ms(g, reps: int = 10, warm: int = 3) -> float:
    """Median duration of one replay of graph `g` over `reps` replays timed one
    by one with HIP events, after `warm` untimed replays."""
    for _ in range(warm):
        g.replay()
    torch.cuda.synchronize()
    ts = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        g.replay()
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1))
    return float(np.median(ts))


def dominant_call_ms(st, reps: int):
    """Duration of one backward call per segment, as in the replayed step:
    the segment's forward runs first, then `reps` back-to-back backward calls
    (nothing between them) are bracketed by one pair of HIP events on the
    launching stream, behind a GPU spin that keeps the host ahead."""
    out = {}
    for s in range(st.wl.T // SEGMENT):
        calls = dict(st.calls(s))
        calls["summaries"]()
        calls["route_attend_fwd"]()
        calls["attend_bwd"]()
        torch.cuda.synchronize()
        t = time.perf_counter()
        calls["attend_bwd"]()
        torch.cuda.synchronize()
        host_ms = (time.perf_counter() - t) * 1e3
        torch.cuda._sleep(_spin_cycles(3.0 * host_ms * reps + 1.0))
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            calls["attend_bwd"]()
        e1.record()
        torch.cuda.synchronize()
        out[s] = e0.elapsed_time(e1) / reps
    return out


def roofline_entry(name, flops, bytes_, ms, traffic=None):
    t = ms * 1e-3
    t_mfma = flops / (BF16_PEAK_TFLOPS * 1e12) if flops else 0.0
    t_hbm = bytes_ / (HBM_PEAK_GBS * 1e9)
    if t_mfma > t_hbm:
        ach = flops / t / 1e12
        return {"kernel": name, "bound": "mfma", "achieved": round(ach, 2), "peak": BF16_PEAK_TFLOPS,
                "unit": "TFLOP/s", "frac": round(ach / BF16_PEAK_TFLOPS, 4), "traffic": traffic}
    ach = bytes_ / t / 1e9
    return {"kernel": name, "bound": "hbm", "achieved": round(ach, 1), "peak": HBM_PEAK_GBS,
            "unit": "GB/s", "frac": round(ach / HBM_PEAK_GBS, 4), "traffic": traffic}


# ----------------------------------------------------------------------------
# Kernel-source fingerprint and the measured HBM traffic of the dominant kernel
# ----------------------------------------------------------------------------

TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hga_attend_bwd_16k_seg1k_hbm_traffic.md")
# The dominant unit of the step: one backward call, i.e. its row-dot kernel
# (D = rowsum(dO * O)) followed by the fused dQ / dK-dV kernel.
DOM_KERNEL = "hga_attend_bwd (bwd_rowdot_kernel + bwd_kernel)"
DOM_PARTS = ("bwd_rowdot_kernel", "bwd_kernel")


def _is_part(name: str, part: str) -> bool:
    """Kernel `name` is the backward part `part` (bwd_kernel also matches the
    combine kernels' names, which are not parts)."""
    return part in name and "combine" not in name


# The sources the backward call is built and launched from.
DOM_SOURCES = ("attend_bwd.hip", "routed_tile.h", "hga_device.h", "hga_kernels.h", "api.hip",
               "../../include/hga.h")


def source_fingerprint() -> str:
    """sha256 over the sources of the dominant kernel (its device code, the
    headers it includes, and the ABI layer that configures its launch): a
    measurement taken on other sources no longer describes the kernel."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2607_15105_amd", "csrc")
    for f in DOM_SOURCES:
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()


# The benchmarked step forms the backward's row term from the bf16 O (no
# float32 copy of O); the traffic record names the variant it measured.
STEP_O_F32 = False


def stored_traffic():
    """Bytes per launch of the dominant kernel from the committed PMC summary,
    or None when there is none, or it was taken on other kernel sources or
    another variant of the step."""
    try:
        text = open(TRAFFIC_FILE).read()
    except OSError:
        return None
    for line in text.splitlines():
        if line.startswith("traffic_json: "):
            rec = json.loads(line[len("traffic_json: "):])
            if (rec.get("fingerprint") == source_fingerprint() and rec.get("o_f32") == STEP_O_F32
                    and rec.get("bwd_kv_parts") == STEP_BWD_KV_PARTS):
                return rec["bytes_per_launch"]
    return None


# ----------------------------------------------------------------------------
# 131K forward (evaluation path)
# ----------------------------------------------------------------------------

def bench_forward(wl: synth.Workload, reps: int):
    """Evaluation-path forward over all T queries of `wl` in one call each:
    summaries, route, routed attention (no float32 O)."""
    hc = hcfg(wl)
    log(f"[bench] generating {wl.T}-token inputs")
    Q, K, V = to_dev(synth.queries(wl)), to_dev(synth.keys(wl)), to_dev(synth.values(wl))
    cs, gs = hga.alloc_summaries(hc, wl.T)
    rb = hga.alloc_route(hc, 0, wl.T)
    O = torch.empty_like(Q)
    lse = torch.empty(wl.T, wl.n_q_heads, device="cuda")

    def calls():
        return [("summaries", lambda: hga.build_summaries(hc, K, 0, wl.T, cs, gs)),
                ("route", lambda: hga.route(hc, Q, 0, cs, gs, rb.sel_chunks, rb.sel_groups,
                                            rb.n_sel_groups, rb.workspace)),
                ("attend_fwd", lambda: hga.attend_fwd(hc, Q, K, V, 0, rb.sel_groups,
                                                      rb.n_sel_groups, O, lse))]
    for _, fn in calls():
        fn()
    torch.cuda.synchronize()
    n_sel = rb.n_sel_groups.cpu().numpy()
    ms, _ = timed_events(calls, reps)
    total = sum(ms.values())
    fl, by, _ = attn_work(wl, 0, wl.T, n_sel, False)  # no float32 O on the evaluation path
    phases = {
        "summaries": {"ms": ms["summaries"], "GB/s": summary_work(wl, 0, wl.T) / ms["summaries"] / 1e6},
        "route": {"ms": ms["route"], "GB/s": route_work(wl, 0, wl.T) / ms["route"] / 1e6},
        "attend_fwd": {"ms": ms["attend_fwd"], "TFLOP/s": fl / ms["attend_fwd"] / 1e9,
                       "GB/s": by / ms["attend_fwd"] / 1e6},
    }
    for p in phases.values():
        for k in list(p):
            p[k] = round(p[k], 3)
    # Dense causal attention on the same inputs and kernels: a sink window
    # covering the whole context and no routed chunks make every block's
    # routed set all earlier tokens.
    wd = dataclasses.replace(wl, top_chunks=0, top_groups=0, sink_tokens=wl.T)
    hd = hcfg(wd)
    zero = torch.zeros_like(rb.n_sel_groups)
    dense = lambda: [("dense_fwd", lambda: hga.attend_fwd(hd, Q, K, V, 0, rb.sel_groups, zero, O, lse))]
    for _, fn in dense():
        fn()
    ms_d, _ = timed_events(dense, max(2, reps // 2))
    fl_d, by_d, _ = attn_work(wd, 0, wl.T, zero.cpu().numpy(), False)
    del Q, K, V, O, cs, gs, rb, lse, zero
    torch.cuda.empty_cache()
    return {"tokens_per_s": round(wl.T / (total * 1e-3), 1), "ms": round(total, 3),
            "selection_density": round(selection_density(wl, 0, wl.T, n_sel), 4),
            "us_per_1k_tokens": round(total * 1e3 / (wl.T / 1024), 2),
            "phases": phases,
            "roofline_attend_fwd": roofline_entry("attend_fwd", fl, by, ms["attend_fwd"]),
            "dense_fwd": {"ms": round(ms_d["dense_fwd"], 3),
                          "TFLOP/s": round(fl_d / ms_d["dense_fwd"] / 1e9, 1),
                          "tokens_per_s": round(wl.T / (ms_d["dense_fwd"] * 1e-3), 1),
                          "hga_speedup": round(ms_d["dense_fwd"] / total, 3)}}


def bench_routing_sweep(reps: int):
    """The 32K routing sweep: the final 2,048-token segment for every (group
    size, top chunks, top groups) point. Phases timed separately: scoring
    (route), the gather alone (hga_gather_routed, compact copies of the routed
    rows), the attention tiles alone (hga_attend_gathered_fwd over those
    copies), the fused gather + attention forward the step uses, and the
    backward."""
    base = synth.WORKLOADS["qwen3_8b_32k_sweep"]
    log(f"[bench] generating {base.T}-token sweep inputs")
    K, V = to_dev(synth.keys(base)), to_dev(synth.values(base))
    t0, n = base.q_begin, base.n_q
    Q = to_dev(synth.queries(base, t0, t0 + n))
    dO = to_dev(synth.grad_output(base, t0, t0 + n))
    O = torch.empty_like(Q)
    lse = torch.empty(n, base.n_q_heads, device="cuda")
    o32 = torch.empty(n, base.n_q_heads, base.head_dim, device="cuda")
    dQ = torch.empty(n, base.n_q_heads, base.head_dim, device="cuda")
    n_act = t0 + n - base.grad_begin
    dK = torch.empty(n_act, base.n_kv_heads, base.head_dim, device="cuda")
    dV = torch.empty_like(dK)
    r_cap = max(hga.gathered_rows(hcfg(base.with_budget(group_size=g, top_chunks=kc, top_groups=kg)))
                for g, kc, kg in synth.SWEEP)
    Kc = torch.empty(n // 64, base.n_kv_heads, r_cap, base.head_dim, dtype=torch.bfloat16, device="cuda")
    Vc = torch.empty_like(Kc)
    O2 = torch.empty_like(O)
    lse2 = torch.empty_like(lse)
    o32b = torch.empty_like(o32)
    points = []
    for g, kc, kg in synth.SWEEP:
        wl = base.with_budget(group_size=g, top_chunks=kc, top_groups=kg)
        hc = hcfg(wl)
        cs, gs = hga.alloc_summaries(hc, wl.T)
        hga.build_summaries(hc, K, 0, wl.T, cs, gs)
        rb = hga.alloc_route(hc, t0, n)
        ws = torch.empty(hga.workspace_size(hc, hga.OP_BWD, t0, n, wl.grad_begin), dtype=torch.uint8,
                         device="cuda")

        # dense [n_qb, Hkv, r_cap, d] views at this point's r_cap
        shp = (n // 64, base.n_kv_heads, hga.gathered_rows(hc), base.head_dim)
        kc_ = Kc.view(-1)[:int(np.prod(shp))].view(shp)
        vc_ = Vc.view(-1)[:int(np.prod(shp))].view(shp)

        def calls():
            return [("route", lambda: hga.route(hc, Q, t0, cs, gs, rb.sel_chunks, rb.sel_groups,
                                                rb.n_sel_groups, rb.workspace)),
                    ("gather", lambda: hga.gather_routed(hc, K, V, t0, n, rb.sel_groups, rb.n_sel_groups,
                                                         kc_, vc_)),
                    ("attend_tiles", lambda: hga.attend_gathered_fwd(hc, Q, kc_, vc_, t0, rb.n_sel_groups,
                                                                     O2, lse2, o32b)),
                    ("attend_fwd", lambda: hga.attend_fwd(hc, Q, K, V, t0, rb.sel_groups, rb.n_sel_groups,
                                                          O, lse, o32)),
                    ("attend_bwd", lambda: hga.attend_bwd(hc, Q, K, V, O, dO, lse, t0, wl.grad_begin,
                                                          rb.sel_groups, rb.n_sel_groups, dQ, dK, dV,
                                                          ws, o32))]
        for _, fn in calls():
            fn()
        torch.cuda.synchronize()
        n_sel = rb.n_sel_groups.cpu().numpy()
        R = routed_sizes(wl, t0, n, n_sel)
        ms, _ = timed_events(calls, reps)
        fl, _, _ = attn_work(wl, t0, n, n_sel, False)
        kv_ws = float(R.sum()) * wl.head_dim * 2 * 2
        gather_bytes = kv_ws + float(np.ceil(R / 64).sum()) * 64 * wl.head_dim * 2 * 2  # read + padded write
        us = lambda k: round(ms[k] * 1e3, 2)
        points.append({"g": g, "k_c": kc, "k_g": kg, "mean_R": round(float(R.mean()), 1),
                       "route_us": us("route"),
                       "route_GBps": round(route_work(wl, t0, n) / (ms["route"] * 1e-3) / 1e9, 1),
                       "gather_us": us("gather"),
                       "gather_GBps": round(gather_bytes / (ms["gather"] * 1e-3) / 1e9, 1),
                       "attend_tiles_us": us("attend_tiles"),
                       "attend_tiles_TFLOPs": round(fl / (ms["attend_tiles"] * 1e-3) / 1e12, 1),
                       "attend_fwd_us": us("attend_fwd"), "attend_bwd_us": us("attend_bwd")})
        del cs, gs, rb, ws
    del K, V, Q, dO, O, lse, o32, dQ, dK, dV, Kc, Vc, O2, lse2, o32b
    torch.cuda.empty_cache()
    return points


# ----------------------------------------------------------------------------
# Tiered storage: history K/V and group summaries in host RAM
# ----------------------------------------------------------------------------

class TieredStep:
    """The 16K training step with tiered storage (Sec. 2.2, Fig. 2): the
    history's exact K/V and the full group-summary table in pinned host
    memory, every chunk summary and a cache of `n_slots` chunks of group
    summaries per kv head in device memory, and each segment's routed rows
    gathered into a compact device working set before its forward and
    backward. The device keeps the K/V of the last `device_segments`
    segments; an older segment's K/V reach the host store on a copy stream
    after its forward, beside the following segments' work, and a segment
    waits for them only before staging its routed rows. Every segment has its
    own routing tables, hit flags and output rows."""

    def __init__(self, wl: synth.Workload, n_slots: int = 256, device_segments: int = 2, o_f32: bool = False):
        self.wl, self.n_slots, self.dev_segs = wl, n_slots, device_segments
        hc = self.hc = step_hcfg(wl)  # the resident step's backward partition
        T, Hkv, d = wl.T, wl.n_kv_heads, wl.head_dim
        n_seg = T // SEGMENT
        log("[bench] tiered step inputs")
        # the synthetic source of each segment's Q/K/V/dO (what a trainer's projections produce)
        self.Kall, self.Vall = to_dev(synth.keys(wl)), to_dev(synth.values(wl))
        self.Qall, self.dOall = to_dev(synth.queries(wl)), to_dev(synth.grad_output(wl))
        torch.cuda.synchronize()
        torch.cuda.reset_peak_memory_stats()
        self.mem0 = torch.cuda.memory_allocated()
        self.K_host = torch.empty(T, Hkv, d, dtype=torch.bfloat16, pin_memory=True)
        self.V_host = torch.empty_like(self.K_host, pin_memory=True)
        self.g_host = torch.zeros(Hkv, d // 4, T // wl.group_size, 4, pin_memory=True)
        self.kh, self.vh = hga.host_view(self.K_host), hga.host_view(self.V_host)
        self.gh = hga.host_view(self.g_host)
        self.hs = hga.Strides(self.K_host.stride(0), self.K_host.stride(1))
        self.group_cap = self.g_host.shape[2]
        self.chunk_sum = torch.zeros(Hkv, d // 4, T // 64, 4, device="cuda")
        self.cache = hga.alloc_group_cache(hc, n_slots, T // 64)
        self.rbs = [hga.alloc_route(hc, s * SEGMENT, SEGMENT) for s in range(n_seg)]
        self.hits = [torch.zeros(SEGMENT // 64, Hkv, max(wl.top_chunks, 1), dtype=torch.int32, device="cuda")
                     for _ in range(n_seg)]
        r_cap = hga.gathered_rows(hc)
        self.Kc = torch.empty(SEGMENT // 64, Hkv, r_cap, d, dtype=torch.bfloat16, device="cuda")
        self.Vc = torch.empty_like(self.Kc)
        self.O = torch.empty(T, wl.n_q_heads, d, dtype=torch.bfloat16, device="cuda")
        self.lse = torch.empty(T, wl.n_q_heads, device="cuda")
        self.o32 = torch.empty(T, wl.n_q_heads, d, device="cuda") if o_f32 else None  # as SegmentedStep
        self.dQ = torch.empty(T, wl.n_q_heads, d, device="cuda")
        self.dK = torch.empty(T, Hkv, d, device="cuda")
        self.dV = torch.empty_like(self.dK)
        self.ws = torch.empty(max(hga.workspace_size(hc, hga.OP_BWD, s * SEGMENT, SEGMENT, s * SEGMENT)
                                  for s in range(n_seg)), dtype=torch.uint8, device="cuda")
        self.copy = torch.cuda.Stream()
        self.ev_fwd = [torch.cuda.Event() for _ in range(n_seg)]
        self.ev_host = [torch.cuda.Event() for _ in range(n_seg)]

    def hist_end(self, s: int) -> int:
        """First token the device still holds while segment s runs."""
        return max(0, (s - self.dev_segs + 1) * SEGMENT)

    def calls(self, s: int):
        hc, wl = self.hc, self.wl
        t0, t1 = s * SEGMENT, (s + 1) * SEGMENT
        he = self.hist_end(s)
        K_act, V_act = self.Kall[he:t1], self.Vall[he:t1]   # the device tier: tokens [he, t1)
        ks = hga.Strides(K_act.stride(0), K_act.stride(1))
        q, do = self.Qall[t0:t1], self.dOall[t0:t1]
        o, l = self.O[t0:t1], self.lse[t0:t1]
        o32 = self.o32[t0:t1] if self.o32 is not None else None
        dq, dk, dv = self.dQ[t0:t1], self.dK[t0:t1], self.dV[t0:t1]
        rb, hit, cache, gh, gc = self.rbs[s], self.hits[s], self.cache, self.gh, self.group_cap
        return [
            ("summaries", lambda: hga.build_summaries_raw(hc, hga.shifted_rows(K_act, he), ks, t0, t1,
                                                          self.chunk_sum, gh, gc)),
            ("route_cached", lambda: hga.route_cached(hc, q, t0, self.chunk_sum, gh, gc, cache, rb.sel_chunks,
                                                      rb.sel_groups, rb.n_sel_groups, hit, rb.workspace)),
            ("cache_update", lambda: hga.group_cache_update(hc, cache, gh, gc, t0, SEGMENT, rb.sel_chunks, hit)),
            ("gather_tiered", lambda: hga.gather_tiered(hc, self.kh, self.vh, self.hs, he, K_act, V_act, t0,
                                                        SEGMENT, rb.sel_groups, rb.n_sel_groups, self.Kc,
                                                        self.Vc)),
            ("attend_fwd", lambda: hga.attend_gathered_fwd(hc, q, self.Kc, self.Vc, t0, rb.n_sel_groups, o, l,
                                                           o32)),
            ("attend_bwd", lambda: hga.attend_gathered_bwd(hc, q, self.Kc, self.Vc, K_act, V_act, he, o, do, l,
                                                           t0, t0, rb.sel_groups, rb.n_sel_groups, dq, dk, dv,
                                                           self.ws, o32)),
        ]

    def detach(self, s: int):
        """Segment s's K/V to the host store."""
        t0, t1 = s * SEGMENT, (s + 1) * SEGMENT
        self.K_host[t0:t1].copy_(self.Kall[t0:t1], non_blocking=True)
        self.V_host[t0:t1].copy_(self.Vall[t0:t1], non_blocking=True)

    def step(self):
        n_seg = self.wl.T // SEGMENT
        main = torch.cuda.current_stream()
        hga.group_cache_clear(self.hc, self.cache)
        self.copy.wait_stream(main)
        for s in range(n_seg):
            for name, fn in self.calls(s):
                if name == "gather_tiered" and s >= self.dev_segs:
                    # the rows this segment reads from the host store have landed
                    main.wait_event(self.ev_host[s - self.dev_segs])
                fn()
                if name == "attend_fwd":
                    self.ev_fwd[s].record(main)
            if s + self.dev_segs < n_seg:  # a later segment reads this one from the host
                with torch.cuda.stream(self.copy):
                    self.copy.wait_event(self.ev_fwd[s])
                    self.detach(s)
                    self.ev_host[s].record(self.copy)
        main.wait_stream(self.copy)


def bench_tier(reps: int, n_slots: int = 256):
    """The tiered 16K step (TieredStep): step time, cache hit rate, the bytes
    that cross the host link and the device memory the step holds."""
    wl = synth.WORKLOADS["qwen3_8b_16k_seg1k"]
    ts = TieredStep(wl, n_slots)
    T, Hkv, d = wl.T, wl.n_kv_heads, wl.head_dim
    ts.step()
    torch.cuda.synchronize()
    # device memory a trainer running this schedule holds: the tiers and the
    # working set, the device window of K/V, and one segment's outputs (the
    # step object keeps every segment's outputs for the tests; a trainer
    # hands each segment's on)
    nb = lambda *xs: sum(x.numel() * x.element_size() for x in xs)
    c = ts.cache
    held = (nb(ts.chunk_sum, c.slot_of, c.slot_chunk, c.cursor, c.groups, ts.Kc, ts.Vc, ts.ws, *ts.hits)
            + sum(nb(rb.sel_chunks, rb.sel_groups, rb.n_sel_groups, rb.workspace) for rb in ts.rbs)
            + 2 * ts.dev_segs * nb(ts.Kall[:SEGMENT])
            + nb(ts.O[:SEGMENT], ts.lse[:SEGMENT], ts.dQ[:SEGMENT], ts.dK[:SEGMENT], ts.dV[:SEGMENT])
            + (nb(ts.o32[:SEGMENT]) if ts.o32 is not None else 0))
    peak_mb = held / 2**20
    hist_rows = miss_chunks = req = n_hit = uniq_rows = 0
    for s in range(T // SEGMENT):
        rb = ts.rbs[s]
        sc, hf = rb.sel_chunks.cpu().numpy(), ts.hits[s].cpu().numpy()
        ok = sc >= 0
        req += int(ok.sum())
        n_hit += int((hf[ok] == 1).sum())
        miss_chunks += int((hf[ok] == 0).sum())
        # routed rows read from the host store: tokens before hist_end, in
        # the sink window, the local window or a selected group, per kv head
        he, t0 = ts.hist_end(s), s * SEGMENT
        b = t0 // 64 + np.arange(SEGMENT // 64)
        ls = np.maximum(0, (b + 1) * 64 - wl.local_tokens)
        sink = np.minimum(wl.sink_tokens, ls)
        win = np.maximum(0, np.minimum(he, (b + 1) * 64) - ls)
        sg = rb.sel_groups.cpu().numpy()
        grp = int(((sg >= 0) & (sg * wl.group_size < he)).sum()) * wl.group_size
        hist_rows += int(np.minimum(sink, he).sum() * Hkv + win.sum() * Hkv + grp)
        # distinct (kv head, token) rows among them: what a segment-wide
        # de-duplicated staging would move over the link
        for h in range(Hkv):
            toks = set()
            for bi, blk in enumerate(b):
                toks.update(range(0, int(min(sink[bi], he))))
                toks.update(range(int(ls[bi]), int(min(he, (blk + 1) * 64))))
                for gid in sg[bi, h]:
                    if gid >= 0 and gid * wl.group_size < he:
                        toks.update(range(int(gid) * wl.group_size, int(gid + 1) * wl.group_size))
            uniq_rows += len(toks)
    # eager on its two streams (as one graph the cross-stream waits cost more)
    ms = eager_median_ms(ts.step, reps)
    ms_graph, g = _graph_ms(ts.step, reps)
    ms_seg, _ = timed_events(lambda: ts.calls(T // SEGMENT - 1), reps)
    del g
    gpc = 64 // wl.group_size
    n_detach = T // SEGMENT - ts.dev_segs
    # history rows the gathers request over the host link (every routed one;
    # rows that several blocks of a call route to are mostly served by the
    # GPU's caches after the first read, so the link carries between the
    # distinct and the routed bytes)
    link = {"history_rows_MB": round(hist_rows * d * 2 * 2 / 1e6, 2),
            "group_summary_misses_MB": round(miss_chunks * gpc * d * 4 / 1e6, 2),
            "detach_MB": round(n_detach * SEGMENT * Hkv * d * 2 * 2 / 1e6, 2),
            "group_summary_writes_MB": round(T // wl.group_size * Hkv * d * 4 / 1e6, 2)}
    total = sum(link.values()) * 1e6
    return {"ms_per_step": round(ms, 4), "ms_per_step_as_one_graph": round(ms_graph, 4), "tokens_per_s": round(T / (ms * 1e-3), 1),
            "cache_slots_per_kv_head": n_slots, "device_segments": ts.dev_segs,
            "history_rows_distinct_per_call_MB": round(uniq_rows * d * 2 * 2 / 1e6, 2),
            "cache_hit_rate": round(n_hit / max(req, 1), 4),
            "host_link_MB_per_step": link, "host_link_GB/s": round(total / (ms * 1e-3) / 1e9, 1),
            # the step's requests over the link against its peak (repeated rows
            # partly served by the GPU's caches, so this is an upper bound)
            "roofline": roofline_obj("host_link", total / (ms * 1e-3) / 1e9, HOST_LINK_PEAK_GBPS, "GB/s"),
            "device_MB_held": round(peak_mb, 1),
            "last_segment_us": {k: round(v * 1e3, 2) for k, v in ms_seg.items()}}


# ----------------------------------------------------------------------------
# HGA against dense causal attention in training (one segment, fwd + bwd)
# ----------------------------------------------------------------------------

def bench_dense_training(reps: int):
    """One training step of a layer over T tokens as one segment (every token
    differentiable), HGA (summaries, routing + forward, backward) against
    dense causal attention (forward and backward over every earlier token,
    the same kernels with a sink window covering the context), at 1K ... 16K.
    The paper's comparison point is whole-model training at 1K and 2K."""
    out = []
    base = synth.WORKLOADS["qwen3_8b_2k"]
    for T in (1024, 2048, 4096, 8192, 16384):
        wl = dataclasses.replace(base, T=T, q_begin=0, n_q=T, grad_begin=0)
        wd = dataclasses.replace(wl, top_chunks=0, top_groups=0, sink_tokens=T)
        hc, hd = hcfg(wl), hcfg(wd)
        log(f"[bench] dense vs HGA training, T={T}")
        Q, K, V, dO = (to_dev(f(wl, 0, T)) for f in (synth.queries, synth.keys, synth.values, synth.grad_output))
        cs, gs = hga.alloc_summaries(hc, T)
        rb = hga.alloc_route(hc, 0, T)
        O = torch.empty_like(Q)
        lse = torch.empty(T, wl.n_q_heads, device="cuda")
        o32 = None  # D from the bf16 O on both sides, as in the segmented step
        dQ = torch.empty(T, wl.n_q_heads, wl.head_dim, device="cuda")
        dK = torch.empty(T, wl.n_kv_heads, wl.head_dim, device="cuda")
        dV = torch.empty_like(dK)
        ws = torch.empty(max(hga.workspace_size(hc, hga.OP_BWD, 0, T, 0), hga.workspace_size(hd, hga.OP_BWD, 0, T, 0)),
                         dtype=torch.uint8, device="cuda")
        zsel = torch.full((T // 64, wl.n_kv_heads, 1), -1, dtype=torch.int32, device="cuda")
        zn = torch.zeros(T // 64, wl.n_kv_heads, dtype=torch.int32, device="cuda")

        def hga_step():
            hga.build_summaries(hc, K, 0, T, cs, gs)
            hga.route_attend_fwd(hc, Q, K, V, 0, cs, gs, rb.sel_chunks, rb.sel_groups, rb.n_sel_groups, O, lse,
                                 rb.workspace, o32)
            hga.attend_bwd(hc, Q, K, V, O, dO, lse, 0, 0, rb.sel_groups, rb.n_sel_groups, dQ, dK, dV, ws, o32)

        def dense_step():
            hga.attend_fwd(hd, Q, K, V, 0, zsel, zn, O, lse, o32)
            hga.attend_bwd(hd, Q, K, V, O, dO, lse, 0, 0, zsel, zn, dQ, dK, dV, ws, o32)
        ms_h, gh = _graph_ms(hga_step, reps)
        n_sel = rb.n_sel_groups.cpu().numpy()
        ms_d, gd = _graph_ms(dense_step, reps)
        fl_d = attn_work(wd, 0, T, zn.cpu().numpy(), False)[0] + attn_work(wd, 0, T, zn.cpu().numpy(), True)[0]
        out.append({"T": T, "hga_ms": round(ms_h, 4), "dense_ms": round(ms_d, 4),
                    "hga_tokens_per_s": round(T / (ms_h * 1e-3), 1),
                    "dense_tokens_per_s": round(T / (ms_d * 1e-3), 1),
                    "hga_over_dense_throughput": round(ms_d / ms_h, 3),
                    "dense_TFLOP/s": round(fl_d / (ms_d * 1e-3) / 1e12, 1),
                    "dense_roofline": roofline_obj("mfma", fl_d / (ms_d * 1e-3) / 1e12, MFMA_BF16_PEAK_TFLOPS,
                                                   "TFLOP/s"),
                    "hga_selection_density": round(selection_density(wl, 0, T, n_sel), 4)})
        del gh, gd, Q, K, V, dO, O, o32, dQ, dK, dV, ws, cs, gs, rb
        torch.cuda.empty_cache()
    return out


# ----------------------------------------------------------------------------
# Per-query routing: decode steps and the strictly causal training step
# ----------------------------------------------------------------------------

HBM_PEAK_GBPS = 8000.0      # MI355X HBM3E
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix
HOST_LINK_PEAK_GBPS = 64.0  # PCIe 5.0 x16, one direction


def roofline_obj(bound: str, achieved: float, peak: float, unit: str, note: str | None = None) -> dict:
    o = {"bound": bound, "achieved": round(achieved, 1), "peak": peak, "unit": unit,
         "frac": round(achieved / peak, 4)}
    if note:
        o["note"] = note
    return o


def rows_bytes(wl, q_begin, n_q, n_sel):
    """Algorithmic bytes of per-query routing + attention over rows
    [q_begin, q_begin + n_q): the call's chunk-summary table once (every
    row's candidates are a prefix of the last row's), each row's chosen
    groups' summaries (float32), its routed K/V rows, its Q and O rows and
    LSE."""
    d, Hkv = wl.head_dim, wl.n_kv_heads
    pos = q_begin + np.arange(n_q)
    end = (pos // 64 + 1) * 64
    ls = np.maximum(0, end - wl.local_tokens)
    sink = np.minimum(wl.sink_tokens, ls)
    n_cand = np.maximum(0, ls // 64 - wl.sink_tokens // 64)
    R = (sink + (pos + 1 - ls))[:, None] + n_sel * wl.group_size
    scan = float(n_cand.max()) * Hkv * d * 4 + n_q * Hkv * wl.top_chunks * (64 // wl.group_size) * d * 4
    kv = float(R.sum()) * d * 2 * 2
    qo = n_q * wl.n_q_heads * (d * 2 * 2 + 4)
    return scan, kv + qo, R


def _graph_ms(fn, reps=10, warm=3):
    """Median duration of one replay of a HIP graph of `fn`."""
    fn()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    return replay_median_ms(g, reps, warm), g


def bench_rows(reps: int):
    """Decode steps with per-query routing at 16K and 131K (one row per call
    and 64 rows per call, timed as graphs of 64 consecutive steps), and the
    16K training step with strictly causal (per-query) routing."""
    out = {"decode": []}
    for name in ("qwen3_8b_16k_seg1k", "qwen3_8b_131k_planted"):
        wl = synth.WORKLOADS[name]
        hc = hcfg(wl)
        T = wl.T
        log(f"[bench] decode inputs {name}")
        K, V = to_dev(synth.keys(wl)), to_dev(synth.values(wl))
        Q = to_dev(synth.queries(wl, T - 64, T))
        cs, gs = hga.alloc_summaries(hc, T)
        hga.build_summaries(hc, K, 0, T, cs, gs)
        sc, sg, ns = hga.alloc_route_rows(hc, 64)
        O = torch.empty_like(Q)
        lse = torch.empty(64, wl.n_q_heads, device="cuda")
        q0 = T - 64

        def steps_one():   # 64 generation steps, one row each
            for r in range(64):
                hga.route_rows(hc, Q[r:r + 1], q0 + r, cs, gs, sc[r:r + 1], sg[r:r + 1], ns[r:r + 1])
                hga.attend_rows_fwd(hc, Q[r:r + 1], K[:q0 + r + 1], V[:q0 + r + 1], q0 + r, sg[r:r + 1],
                                    ns[r:r + 1], O[r:r + 1], lse[r:r + 1])

        def step_block():  # the same 64 rows in one call (chunked or speculative decode)
            hga.route_rows(hc, Q, q0, cs, gs, sc, sg, ns)
            hga.attend_rows_fwd(hc, Q, K, V, q0, sg, ns, O, lse)
        ms1, g1 = _graph_ms(steps_one, reps)
        ms64, g64 = _graph_ms(step_block, reps)
        n_sel = ns.cpu().numpy()
        scan, kvqo, R = rows_bytes(wl, q0, 64, n_sel)
        gb1 = (scan + kvqo) / (ms1 * 1e-3) / 1e9
        gb64 = (scan + kvqo) / (ms64 * 1e-3) / 1e9
        out["decode"].append({
            "T": T, "rows_per_call": 1, "us_per_step": round(ms1 * 1e3 / 64, 2),
            "tokens_per_s": round(64 / (ms1 * 1e-3), 1),
            "GB/s": round(gb1, 1), "mean_R": round(float(R.mean()), 1),
            # one row per step reads ~1 MB: the two launches' latency, not HBM, bounds it
            "roofline": roofline_obj("hbm", gb1, HBM_PEAK_GBPS, "GB/s", note="latency-bound (two launches per step)")})
        out["decode"].append({
            "T": T, "rows_per_call": 64, "us_per_call": round(ms64 * 1e3, 2),
            "tokens_per_s": round(64 / (ms64 * 1e-3), 1),
            "GB/s": round(gb64, 1), "roofline": roofline_obj("hbm", gb64, HBM_PEAK_GBPS, "GB/s")})
        del g1, g64, K, V, Q, cs, gs, O
        torch.cuda.empty_cache()

    # the 16K training step with per-query routing (the strictly causal variant)
    wl = synth.WORKLOADS["qwen3_8b_16k_seg1k"]
    hc = hcfg(wl)
    T = wl.T
    Q, K, V, dO = (to_dev(f(wl, 0, T)) for f in (synth.queries, synth.keys, synth.values, synth.grad_output))
    cs, gs = hga.alloc_summaries(hc, T)
    sc, sg, ns = hga.alloc_route_rows(hc, SEGMENT)
    O = torch.empty_like(Q)
    lse = torch.empty(T, wl.n_q_heads, device="cuda")
    o32 = None  # D from the bf16 O, as in the segmented step
    dQ = torch.empty(SEGMENT, wl.n_q_heads, wl.head_dim, device="cuda")
    dK = torch.empty(SEGMENT, wl.n_kv_heads, wl.head_dim, device="cuda")
    dV = torch.empty_like(dK)
    ws = torch.empty(hga.rows_workspace_size(hc, SEGMENT), dtype=torch.uint8, device="cuda")

    def calls(s):
        t0, t1 = s * SEGMENT, (s + 1) * SEGMENT
        q, o, l, do = Q[t0:t1], O[t0:t1], lse[t0:t1], dO[t0:t1]
        return [("summaries", lambda: hga.build_summaries(hc, K, t0, t1, cs, gs)),
                ("route_rows", lambda: hga.route_rows(hc, q, t0, cs, gs, sc, sg, ns)),
                ("attend_rows_fwd", lambda: hga.attend_rows_fwd(hc, q, K, V, t0, sg, ns, o, l, o32)),
                ("attend_rows_bwd", lambda: hga.attend_rows_bwd(hc, q, K, V, o, do, l, t0, t0, sg, ns, dQ, dK,
                                                                dV, ws, o32))]

    def step():
        for s in range(T // SEGMENT):
            for _, fn in calls(s):
                fn()
    ms_step, g = _graph_ms(step, reps)
    ms_last, _ = timed_events(lambda: calls(T // SEGMENT - 1), reps)
    del g
    # algorithmic bytes of the last segment's calls: routing reads each row's
    # candidate summaries and its Q; the forward the routed K/V rows, Q, O and
    # LSE; the backward those again with dO, plus dQ and dK/dV (float32)
    t0 = T - SEGMENT
    scan, kvqo, _ = rows_bytes(wl, t0, SEGMENT, ns.cpu().numpy())
    q_b = SEGMENT * wl.n_q_heads * wl.head_dim * 2
    by = {"route_rows": scan + q_b, "attend_rows_fwd": kvqo,
          "attend_rows_bwd": kvqo + q_b + SEGMENT * wl.n_q_heads * wl.head_dim * 4
          + SEGMENT * wl.n_kv_heads * wl.head_dim * 4 * 2}
    roof = {k: roofline_obj("hbm", by[k] / (ms_last[k] * 1e-3) / 1e9, HBM_PEAK_GBPS, "GB/s")
            for k in by if k in ms_last}
    out["strict_causal_16k"] = {
        "ms_per_step": round(ms_step, 4), "tokens_per_s": round(T / (ms_step * 1e-3), 1),
        "last_segment_us": {k: round(v * 1e3, 2) for k, v in ms_last.items()},
        "last_segment_roofline": roof,
        "note": "every query routed on its own (per-query descriptor, block windows): no query's "
                "attended set depends on a later query"}
    return out


# ----------------------------------------------------------------------------
# CPU oracle baseline (bounded sample)
# ----------------------------------------------------------------------------

def _cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _oracle_segments(orc, cfg, wl, segs, K, V):
    """The oracle's summaries + route + fwd + bwd over the given segments; the
    seconds it took and its routing per segment."""
    routing, t_total = {}, 0.0
    for s in segs:
        t0 = s * SEGMENT
        Q = synth.queries(wl, t0, t0 + SEGMENT)
        dO = synth.grad_output(wl, t0, t0 + SEGMENT)
        t = time.perf_counter()
        c, g = orc.summaries(K, cfg, t0 + SEGMENT)
        r = orc.route(Q, c, g, cfg, t0, SEGMENT)
        orc.attend_fwd(Q, K, V, cfg, t0, SEGMENT, r.sel_groups, r.n_sel_groups)
        orc.attend_bwd(Q, K, V, dO, cfg, t0, SEGMENT, t0, r.sel_groups, r.n_sel_groups)
        t_total += time.perf_counter() - t
        routing[s] = (r, g, Q)
    return t_total, routing


def cpu_baseline(wl: synth.Workload, gpu_routing=None, one_thread_segments: int = 2):
    """The oracle as it stands (float64 NumPy, test infrastructure) on the
    host cores over the whole 16K workload, then on a single thread over its
    last segments. With the GPU's routing of the same segments it also counts
    how the two routings agree: exact, near-ties (the rule of the parity
    tests) and mismatches."""
    from threadpoolctl import threadpool_info, threadpool_limits

    from oracle import hga_oracle as orc
    avail = len(os.sched_getaffinity(0))
    cfg = orc.Config(wl.n_q_heads, wl.n_kv_heads, wl.head_dim, wl.chunk_size, wl.group_size,
                     wl.query_block, wl.top_chunks, wl.top_groups, wl.sink_tokens, wl.local_tokens)
    n_seg = wl.T // SEGMENT
    K, V = synth.keys(wl), synth.values(wl)
    with threadpool_limits(limits=avail):
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
        t_all, routing = _oracle_segments(orc, cfg, wl, range(n_seg), K, V)
    last = list(range(n_seg - one_thread_segments, n_seg))
    with threadpool_limits(limits=1):
        t_one, _ = _oracle_segments(orc, cfg, wl, last, K, V)
    out = {"value": round(wl.T / t_all, 2), "unit": "query tokens/s", "cores": min(threads, avail),
           "kind": "oracle",
           "sample": f"all 16 segments of the 16K workload ({wl.T} query tokens): summaries + route + "
                     f"fwd + bwd, float64 NumPy with Python loops over (block, head), {t_all:.1f} s; "
                     f"BLAS pool of {threads} threads (the Python loops run on one)",
           "host_cpus": avail, "cpu_model": _cpu_model(),
           "one_thread": {"value": round(len(last) * SEGMENT / t_one, 2), "unit": "query tokens/s",
                          "sample": f"segments {last[0]}..{last[-1]} on one thread, {t_one:.1f} s"}}
    if gpu_routing:
        from tests import parity as P
        tally = {"exact": 0, "near_ties": 0, "mismatches": 0}
        for s, (r, g, Q) in routing.items():
            sc, sg, ns = gpu_routing[s]
            ws = dataclasses.replace(wl, T=(s + 1) * SEGMENT, q_begin=s * SEGMENT, n_q=SEGMENT,
                                     grad_begin=s * SEGMENT)
            run = P.GpuRun(None, None, sc, sg, ns, None, None)
            rep = P.compare_routing(ws, run, r, g, Q)
            for k in tally:
                tally[k] += getattr(rep, k)
        out["routing_vs_oracle"] = dict(tally, pairs=sum(tally.values()),
                                        rule="near-tie: differing index within 1e-5 relative of the "
                                             "oracle's k-th float64 score")
    return out


# ----------------------------------------------------------------------------
# Profile support: a short pass for rocprofv3 --pmc, and the summaries kept
# under profiles/
# ----------------------------------------------------------------------------

CALIB_BYTES = 256 << 20


def pmc_pass(st):
    """A plain copy of known size (the counter calibration), then one eager
    step of the 16K workload after a warm-up step."""
    src = torch.ones(CALIB_BYTES // 4, device="cuda")
    dst = torch.empty_like(src)
    st.step()
    torch.cuda.synchronize()
    torch.mul(src, 2.0, out=dst)   # reads CALIB_BYTES, writes CALIB_BYTES
    torch.cuda.synchronize()
    st.step()
    torch.cuda.synchronize()
    log("[bench] pmc pass done")


def pmc_fwd131k_pass():
    """The calibration copy, then the 131K evaluation forward (summaries,
    route, routed attention) once after a warm-up, for rocprofv3 --pmc. Prints
    the calls' algorithmic bytes as one `work_json:` line."""
    wl = synth.WORKLOADS["qwen3_8b_131k_planted"]
    hc = hcfg(wl)
    Q, K, V = to_dev(synth.queries(wl)), to_dev(synth.keys(wl)), to_dev(synth.values(wl))
    cs, gs = hga.alloc_summaries(hc, wl.T)
    rb = hga.alloc_route(hc, 0, wl.T)
    O = torch.empty_like(Q)
    lse = torch.empty(wl.T, wl.n_q_heads, device="cuda")

    def fwd():
        hga.build_summaries(hc, K, 0, wl.T, cs, gs)
        hga.route(hc, Q, 0, cs, gs, rb.sel_chunks, rb.sel_groups, rb.n_sel_groups, rb.workspace)
        hga.attend_fwd(hc, Q, K, V, 0, rb.sel_groups, rb.n_sel_groups, O, lse)
    fwd()
    torch.cuda.synchronize()
    src = torch.ones(CALIB_BYTES // 4, device="cuda")
    dst = torch.empty_like(src)
    torch.mul(src, 2.0, out=dst)   # reads CALIB_BYTES, writes CALIB_BYTES
    torch.cuda.synchronize()
    fwd()
    torch.cuda.synchronize()
    n_sel = rb.n_sel_groups.cpu().numpy()
    _, by, _ = attn_work(wl, 0, wl.T, n_sel, False)  # no float32 O on the evaluation path
    print("work_json: " + json.dumps({"summaries": summary_work(wl, 0, wl.T), "route": route_work(wl, 0, wl.T),
                                      "attend_fwd": by}), flush=True)
    log("[bench] 131K forward pmc pass done")


FWD_KERNELS = (("summaries", "summaries_kernel"), ("route", "route_kernel"), ("attend_fwd", "attend_fwd_kernel"))


def summarize_pmc_fwd(fetch_db, write_db, work_log, out, command):
    """HBM bytes of each kernel of the 131K evaluation forward (the last
    dispatch of each), scaled by the calibration copy, beside its algorithmic
    bytes."""
    work = None
    for line in open(work_log):
        if line.startswith("work_json: "):
            work = json.loads(line[len("work_json: "):])
    res = {}
    for label, db, counter in (("fetch", fetch_db, "FETCH_SIZE"), ("write", write_db, "WRITE_SIZE")):
        rows = _pmc_per_dispatch(db, counter)
        calib = max(v for n, v in rows if "Mul" in n or "mul" in n)        # KiB
        scale = (CALIB_BYTES / 1024.0) / calib
        res[label] = {"calib_kib": calib, "scale": scale}
        for name, part in FWD_KERNELS:
            res[label][name] = [v for n, v in rows if part in n][-1] * 1024.0 * scale
    lines = ["# HBM traffic of the 131K evaluation forward: summaries, route, routed attention (bench.py)", "",
             "Commands (run from the repository root), one counter per run:", "", "```", command, "```", "",
             f"Calibration: a plain elementwise copy of {CALIB_BYTES >> 20} MiB (read and written once) "
             f"reads FETCH_SIZE {res['fetch']['calib_kib']:.0f} KiB and WRITE_SIZE "
             f"{res['write']['calib_kib']:.0f} KiB; each kernel's counter is scaled by "
             f"{CALIB_BYTES >> 10} KiB over that reading. Algorithmic bytes as in bench.py "
             "(route: query rows, the candidate chunk summaries once per kv head and the selected chunks' "
             "group summaries; attend_fwd: the gathered K/V working set, Q, O and LSE). The two counters "
             "count what the L2 fetches from and writes to the memory fabric (Infinity Cache or HBM): bytes "
             "that neighbouring blocks share through the L2 or the Infinity Cache are counted once, so a "
             "ratio below 1 means reuse, not skipped work.", "",
             "| kernel | fetched MB | written MB | HBM MB | algorithmic MB | HBM / algorithmic |",
             "|---|---|---|---|---|---|"]
    for name, _ in FWD_KERNELS:
        f, w = res["fetch"][name], res["write"][name]
        alg = work[name] if work else float("nan")
        lines.append(f"| {name} | {f / 1e6:.1f} | {w / 1e6:.1f} | {(f + w) / 1e6:.1f} | {alg / 1e6:.1f} | "
                     f"{(f + w) / alg:.2f} |")
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def pmc_mfma_pass():
    """The 32K routing sweep's point (g 8, k_c 8, k_g 32) over its final
    2,048-token segment, each kernel once after a warm-up: routing, the gather
    alone, the attention tiles over the compact rows (no float32 O), the fused
    forward with float32 O, and the backward. For rocprofv3 --pmc with the
    MFMA counters."""
    wl = synth.WORKLOADS["qwen3_8b_32k_sweep"].with_budget(group_size=8, top_chunks=8, top_groups=32)
    hc = hcfg(wl)
    t0, n = wl.q_begin, wl.n_q
    K, V = to_dev(synth.keys(wl)), to_dev(synth.values(wl))
    Q = to_dev(synth.queries(wl, t0, t0 + n))
    dO = to_dev(synth.grad_output(wl, t0, t0 + n))
    O, O2 = torch.empty_like(Q), torch.empty_like(Q)
    lse, lse2 = (torch.empty(n, wl.n_q_heads, device="cuda") for _ in range(2))
    o32 = torch.empty(n, wl.n_q_heads, wl.head_dim, device="cuda")
    dQ = torch.empty_like(o32)
    dK = torch.empty(n, wl.n_kv_heads, wl.head_dim, device="cuda")
    dV = torch.empty_like(dK)
    cs, gs = hga.alloc_summaries(hc, wl.T)
    rb = hga.alloc_route(hc, t0, n)
    Kc = torch.empty(n // 64, wl.n_kv_heads, hga.gathered_rows(hc), wl.head_dim, dtype=torch.bfloat16,
                     device="cuda")
    Vc = torch.empty_like(Kc)
    ws = torch.empty(hga.workspace_size(hc, hga.OP_BWD, t0, n, t0), dtype=torch.uint8, device="cuda")
    hga.build_summaries(hc, K, 0, wl.T, cs, gs)
    for _ in range(2):
        hga.route(hc, Q, t0, cs, gs, rb.sel_chunks, rb.sel_groups, rb.n_sel_groups, rb.workspace)
        hga.gather_routed(hc, K, V, t0, n, rb.sel_groups, rb.n_sel_groups, Kc, Vc)
        hga.attend_gathered_fwd(hc, Q, Kc, Vc, t0, rb.n_sel_groups, O2, lse2)
        hga.attend_fwd(hc, Q, K, V, t0, rb.sel_groups, rb.n_sel_groups, O, lse, o32)
        hga.attend_bwd(hc, Q, K, V, O, dO, lse, t0, t0, rb.sel_groups, rb.n_sel_groups, dQ, dK, dV, ws, o32)
        torch.cuda.synchronize()
    log("[bench] mfma pmc pass done")


def summarize_mfma(db, out, command):
    """MFMA counters per kernel of the MFMA pass (last dispatch of each):
    executed bf16 MFMA work (32x32x16 instructions x 32,768 flops) over the
    dispatch duration, and SQ_VALU_MFMA_BUSY_CYCLES over the 1,024 SIMDs'
    cycles at 2.4 GHz."""
    import sqlite3
    con = sqlite3.connect(db)
    dur = {d: t for d, t in con.execute("select dispatch_id, duration from kernels")}
    vals = {}
    for name, disp, cn, v in con.execute(
            "select kernel_name, dispatch_id, counter_name, value from counters_collection"):
        vals.setdefault(name, {}).setdefault(disp, {}).setdefault(cn, 0.0)
        vals[name][disp][cn] += v
    lines = ["# MFMA counters of the attention kernels: 32K sweep point g 8, k_c 8, k_g 32, "
             "final 2,048-token segment (bench.py --pmc-mfma)", "",
             "Command (run from the repository root):", "", "```", command, "```", "",
             "Last dispatch of each kernel. `MFMA TFLOP/s` = SQ_INSTS_MFMA x 32,768 flops (one "
             "32x32x16 bf16 instruction) / duration: executed matrix work, including the masked "
             "parts of diagonal and padding tiles and, with a float32 O, the second (lo) P.V "
             "product. `MFMA busy` = SQ_VALU_MFMA_BUSY_CYCLES / (1,024 SIMDs x duration x 2.4 GHz).",
             "", "| kernel | us | SQ_INSTS_MFMA | MFMA TFLOP/s | of 2,500 | MFMA busy |",
             "|---|---|---|---|---|---|"]
    for name, per in vals.items():
        if not name.startswith("_ZN3hga") and "hga" not in name:
            continue
        disp = max(per)
        c = per[disp]
        us = dur.get(disp, 0) / 1e3
        if us <= 0 or "SQ_INSTS_MFMA" not in c:
            continue
        tf = c["SQ_INSTS_MFMA"] * 32768 / (us * 1e-6) / 1e12
        busy = c.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) / (1024 * us * 1e-6 * 2.4e9)
        lines.append(f"| `{_short(name)[:80]}` | {us:.1f} | {int(c['SQ_INSTS_MFMA'])} | {tf:.1f} | "
                     f"{tf / BF16_PEAK_TFLOPS:.3f} | {busy:.3f} |")
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def _short(name):
    import re
    import subprocess
    try:
        name = subprocess.run(["c++filt", name], capture_output=True, text=True).stdout.strip() or name
    except OSError:
        pass
    return re.sub(r"\(hga::\w+\)|hga::", "", name)


def summarize_trace(db, out, command, title=None, step_section=True):
    import sqlite3
    con = sqlite3.connect(db)
    rows = list(con.execute(
        "select name, count(*), sum(duration)/1e3, avg(duration)/1e3, min(duration)/1e3, max(duration)/1e3, "
        "max(grid_x), max(workgroup_x), max(vgpr_count), max(accum_vgpr_count), max(lds_size) "
        "from kernels group by name order by sum(duration) desc"))
    tot = sum(r[2] for r in rows)
    lines = [f"# Kernel trace: {title or '16K segmented fwd+bwd step (bench.py)'}", "",
             "Command (run from the repository root):", "", "```", command, "```", "",
             "rocprofv3 kernel trace of every dispatch of the run; durations in microseconds.", "",
             "| kernel | calls | total us | avg us | min us | max us | % | grid | wg | vgpr | agpr | lds B |",
             "|---|---|---|---|---|---|---|---|---|---|---|---|"]
    for r in rows:
        name = _short(r[0])
        name = name if len(name) <= 90 else name[:87] + "..."
        lines.append(f"| `{name}` | {r[1]} | {r[2]:.1f} | {r[3]:.2f} | {r[4]:.2f} | {r[5]:.2f} | "
                     f"{100 * r[2] / tot:.1f} | {r[6]} | {r[7]} | {r[8]} | {r[9]} | {r[10]} |")
    # the dominant kernel per segment of the 16K step (all its dispatches are
    # that workload's backward calls, sixteen per step in segment order)
    ks = list(con.execute("select name, duration from kernels where name like '%bwd_%' order by start")) \
        if step_section else []
    parts = [[d / 1e3 for n, d in ks if _is_part(n, p)] for p in DOM_PARTS]
    d = [sum(x) for x in zip(*parts)]  # per backward call, in call order
    if d:
        # every backward dispatch of the run belongs to the 16K step, sixteen
        # calls per pass in segment order; the median per segment is that of
        # the graph replays and back-to-back timed calls, which are most of
        # them (the eagerly timed phase passes run with the profiler between
        # dispatches and take longer)
        per = np.array(d[: len(d) // 16 * 16]).reshape(-1, 16)
        med = np.median(per, axis=0)
        lines += ["", f"`{DOM_KERNEL}` by segment of the 16K step (median over {per.shape[0]} passes, us):", "",
                  "| segment | " + " | ".join(str(i) for i in range(16)) + " |",
                  "|---" * 17 + "|",
                  "| us | " + " | ".join(f"{v:.1f}" for v in med) + " |"]
        wl = synth.WORKLOADS["qwen3_8b_16k_seg1k"]
        segs = unsplit_bwd_segments(step_hcfg(wl))
        lines += ["", f"Backward calls without a split of the dK/dV work (segments {segs[0]}..{segs[-1]}): "
                  f"{med[segs].mean():.2f} us per call ({' + '.join(DOM_PARTS)}), the mean of their medians."]
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def _pmc_per_dispatch(db, counter):
    import sqlite3
    con = sqlite3.connect(db)
    vals = {}
    for name, disp, v in con.execute(
            "select kernel_name, dispatch_id, value from counters_collection where counter_name = ?", (counter,)):
        key = (disp, name)
        vals[key] = vals.get(key, 0.0) + v
    return [(name, v) for (disp, name), v in sorted(vals.items())]


def summarize_pmc(fetch_db, write_db, out, command):
    """HBM bytes per backward call (row-dot + main kernel) over the segments
    whose dK/dV work is not split, each counter scaled by what it reads for
    the calibration copy (CALIB_BYTES read and written)."""
    wl = synth.WORKLOADS["qwen3_8b_16k_seg1k"]
    segs = unsplit_bwd_segments(step_hcfg(wl))
    res = {}
    for label, db, counter in (("fetch", fetch_db, "FETCH_SIZE"), ("write", write_db, "WRITE_SIZE")):
        rows = _pmc_per_dispatch(db, counter)
        calib = max(v for n, v in rows if "Mul" in n or "mul" in n)        # KiB
        per_part = [[v for n, v in rows if _is_part(n, p)][-16:] for p in DOM_PARTS]  # the measured step
        bwd = [sum(x) for x in zip(*per_part)]                            # per backward call
        scale = (CALIB_BYTES / 1024.0) / calib
        res[label] = {"calib_kib": calib, "scale": scale,
                      "per_segment_kib": bwd,
                      "bytes_per_launch": float(np.mean([bwd[s] for s in segs])) * 1024.0 * scale}
    total = res["fetch"]["bytes_per_launch"] + res["write"]["bytes_per_launch"]
    rec = {"kernel": DOM_KERNEL, "segments": f"{segs[0]}..{segs[-1]}", "bytes_per_launch": round(total),
           "fetch_bytes": round(res["fetch"]["bytes_per_launch"]),
           "write_bytes": round(res["write"]["bytes_per_launch"]),
           "fetch_scale": round(res["fetch"]["scale"], 4), "write_scale": round(res["write"]["scale"], 4),
           "o_f32": STEP_O_F32, "bwd_kv_parts": STEP_BWD_KV_PARTS, "fingerprint": source_fingerprint()}
    lines = ["# HBM traffic of one backward call (bwd_rowdot_kernel + bwd_kernel): 16K segmented step (bench.py)", "",
             "Commands (run from the repository root), one counter per run:", "", "```", command, "```", "",
             f"Calibration: a plain elementwise copy of {CALIB_BYTES >> 20} MiB (read and written once) "
             f"reads FETCH_SIZE {res['fetch']['calib_kib']:.0f} KiB and WRITE_SIZE "
             f"{res['write']['calib_kib']:.0f} KiB; each counter of the backward kernels is scaled by "
             f"{CALIB_BYTES >> 10} KiB over that reading.", "",
             "| segment | " + " | ".join(str(i) for i in range(16)) + " |", "|---" * 17 + "|",
             "| FETCH_SIZE KiB | " + " | ".join(f"{v:.0f}" for v in res["fetch"]["per_segment_kib"]) + " |",
             "| WRITE_SIZE KiB | " + " | ".join(f"{v:.0f}" for v in res["write"]["per_segment_kib"]) + " |", "",
             f"Per call over the segments without a split of the dK/dV work, {rec['segments']}: "
             f"{rec['fetch_bytes'] / 1e6:.2f} MB fetched + {rec['write_bytes'] / 1e6:.2f} MB written "
             f"= {total / 1e6:.2f} MB.", "",
             "The line below is read by bench.py (roofline.traffic) while the kernel sources keep this "
             "fingerprint:", "",
             "traffic_json: " + json.dumps(rec)]
    open(out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


# ----------------------------------------------------------------------------

def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-131k", action="store_true")
    ap.add_argument("--no-sweep", action="store_true", help="skip the 32K routing sweep")
    ap.add_argument("--no-rows", action="store_true", help="skip the per-query routing (decode) measurements")
    ap.add_argument("--no-dense", action="store_true", help="skip the HGA-vs-dense training comparison")
    ap.add_argument("--no-tier", action="store_true", help="skip the tiered (host RAM history) step")
    ap.add_argument("--event-reps", type=int, default=10)
    ap.add_argument("--part", choices=("context", "sweep", "rows", "dense", "tier"),
                    help="(internal) one further configuration, run in a fresh process by the main run")
    ap.add_argument("--context-T", type=int, default=131072)
    ap.add_argument("--pmc-pass", action="store_true",
                    help="one eager 16K step plus a 256 MiB calibration copy, for rocprofv3 --pmc")
    ap.add_argument("--summarize-trace", metavar="DB",
                    help="write the kernel-trace summary of a rocprofv3 results database to --out")
    ap.add_argument("--pmc-mfma", action="store_true",
                    help="the attention kernels of one 32K sweep point, for rocprofv3 --pmc (MFMA counters)")
    ap.add_argument("--summarize-mfma", metavar="DB",
                    help="write the MFMA counters of a --pmc-mfma run to --out")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DB", "WRITE_DB"),
                    help="write the HBM traffic of the dominant kernel from two PMC passes to --out")
    ap.add_argument("--pmc-fwd131k", action="store_true",
                    help="the 131K evaluation forward plus the calibration copy, for rocprofv3 --pmc")
    ap.add_argument("--summarize-pmc-fwd", nargs=3, metavar=("FETCH_DB", "WRITE_DB", "WORK_LOG"),
                    help="write the HBM traffic of the 131K forward's kernels to --out")
    ap.add_argument("--command", default="", help="command line recorded in a summary")
    ap.add_argument("--title", default=None, help="title of a kernel-trace summary")
    ap.add_argument("--no-step-section", action="store_true",
                    help="kernel-trace summary of a run that is not the 16K step (no per-segment table)")
    ap.add_argument("--out", help="summary file")
    args = ap.parse_args()
    if args.summarize_trace:
        summarize_trace(args.summarize_trace, args.out, args.command, args.title, not args.no_step_section)
        return
    if args.summarize_pmc:
        summarize_pmc(*args.summarize_pmc, args.out, args.command)
        return
    if args.summarize_mfma:
        summarize_mfma(args.summarize_mfma, args.out, args.command)
        return
    if args.summarize_pmc_fwd:
        summarize_pmc_fwd(*args.summarize_pmc_fwd, args.out, args.command)
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures the HGA hot path on one GPU only; runs on more than one GPU are "
              "not implemented.", file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    hga.lib()
    if args.pmc_mfma:
        pmc_mfma_pass()
        return
    if args.pmc_fwd131k:
        pmc_fwd131k_pass()
        return
    if args.part:
        main_part(args)
        return

    wl = synth.WORKLOADS["qwen3_8b_16k_seg1k"]
    torch.cuda.reset_peak_memory_stats()
    mem0 = torch.cuda.memory_allocated()
    st = SegmentedStep(wl, o_f32=STEP_O_F32)
    st.record_routing()
    peak_mb = (torch.cuda.max_memory_allocated() - mem0) / 2**20
    work, bwd_work = st.work()
    if args.pmc_pass:
        pmc_pass(st)
        return

    # One full step (48 ABI calls) launched eagerly on its two streams. As
    # one HIP graph the same step runs slower: the graph's two branches are
    # spread over several hardware queues, and every dependency between
    # them (each segment's forward to its backward and to the next
    # summaries) waits ~10 us, where an eager cross-stream wait costs little.
    for _ in range(args.warmup):
        st.step()
    torch.cuda.synchronize()
    t = time.perf_counter()
    for _ in range(args.steps):
        st.step()
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t) * 1e3 / args.steps
    value = wl.T / (ms_step * 1e-3)
    ms_step_median = eager_median_ms(st.step, 10, 3)
    # the same step as one graph, and its calls in one stream, for comparison
    ms_graph, g = _graph_ms(st.step, 10)
    del g
    st.overlap = False
    ms_seq, g_seq = _graph_ms(st.step, 10)
    ms_seq_eager = eager_median_ms(st.step, 10, 3)
    st.overlap = True
    del g_seq
    # the same step with the optional float32 copy of O (D from it), for reference
    st32 = SegmentedStep(wl, o_f32=True)
    st32.step()
    ms_f32 = eager_median_ms(st32.step, 10, 3)
    del st32
    torch.cuda.empty_cache()

    # eager per-call durations over the same step (the backward per segment)
    def step_calls():
        return [(f"{n}#{s}", fn) for s in range(wl.T // SEGMENT) for n, fn in st.calls(s)]
    ms_seg, cnt_seg = timed_events(step_calls, args.event_reps)
    bwd_seg = {int(k.split("#")[1]): v for k, v in ms_seg.items() if k.startswith("attend_bwd#")}
    fwd_seg = {int(k.split("#")[1]): v for k, v in ms_seg.items() if k.startswith("route_attend_fwd#")}
    sum_seg = {int(k.split("#")[1]): v for k, v in ms_seg.items() if k.startswith("summaries#")}
    n_seg = wl.T // SEGMENT
    ms_call = {"summaries": float(np.mean(list(sum_seg.values()))),
               "route_attend_fwd": float(np.mean(list(fwd_seg.values()))),
               "attend_bwd": float(np.mean(list(bwd_seg.values())))}
    per_step = {k: ms_call[k] * n_seg for k in ms_call}
    eager_ms = sum(per_step.values())
    phases = {}
    for k in ("summaries", "route_attend_fwd", "attend_bwd"):
        fl, by, im = work[k]
        phases[k] = {"ms_per_step": round(per_step[k], 4), "us_per_call": round(ms_call[k] * 1e3, 2),
                     "GB/s": round(by / (per_step[k] * 1e-3) / 1e9, 1)}
        if im:
            phases[k]["impl_GB/s"] = round((by + im) / (per_step[k] * 1e-3) / 1e9, 1)
        if fl:
            phases[k]["TFLOP/s"] = round(fl / (per_step[k] * 1e-3) / 1e12, 2)
    # Roofline of the dominant unit, one backward call (row-dot kernel + the
    # fused dQ / dK-dV kernel), over the segments whose dK/dV work is not
    # split (split calls add a combine kernel): every segment of the step,
    # which never splits.
    segs = st.single_kernel_bwd_segments()
    fl = float(np.mean([bwd_work[s][0] for s in segs]))
    by = float(np.mean([bwd_work[s][1] for s in segs]))
    im = float(np.mean([bwd_work[s][2] for s in segs]))
    dom_ms = dominant_call_ms(st, args.event_reps * 2)
    ms_dom = float(np.mean([v for s, v in dom_ms.items() if s in segs]))
    traffic = stored_traffic()
    roof = roofline_entry(DOM_KERNEL, fl, by, ms_dom, traffic)
    roof.update({"segments": f"{segs[0]}..{segs[-1]}", "us_per_call": round(ms_dom * 1e3, 2),
                 "algorithmic_bytes_per_call": round(by), "flops_per_call": round(fl),
                 "impl_bytes_per_call": round(im),
                 "impl_note": "bytes beyond the method's (none without the optional float32 copy of O)",
                 "traffic_over_algorithmic": round(traffic / by, 3) if traffic else None})
    # the same over segments 4..15, whose calls have enough routable history
    # that the library's default would not split them either (the set the
    # figure was taken over while the step split segments 0..3)
    late = [s for s in segs if s >= 4]
    by_l = float(np.mean([bwd_work[s][1] for s in late]))
    ms_l = float(np.mean([dom_ms[s] for s in late]))
    roof["segments_4_15"] = {"us_per_call": round(ms_l * 1e3, 2), "algorithmic_bytes_per_call": round(by_l),
                             "achieved": round(by_l / (ms_l * 1e-3) / 1e9, 1),
                             "frac": round(by_l / (ms_l * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4)}

    out = {"metric": METRIC, "value": round(value, 1), "unit": "query tokens/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
           "data": "synthetic",
           "config": {"workload": "qwen3_8b_16k_seg1k: one Qwen3-8B attention layer (Hq 32, Hkv 8, "
                                  "d 128) over 16,384 tokens as 16 x 1,024-token segments, "
                                  "summaries + route + fwd + bwd per segment; chunk 64, group 8, "
                                  "top 8 chunks / 16 groups, sink 64, local 128",
                      "global_batch": 1, "seq_len": wl.T, "parallelism": "single GPU"},
           "roofline": roof,
           "ms_per_step_median_of_10": round(ms_step_median, 4),
           "ms_per_step_as_one_graph": round(ms_graph, 4),
           "ms_per_step_with_f32_O": round(ms_f32, 4),
           "numerics": "bf16 inputs, float32 accumulation; D = rowsum(dO * O) over the bf16 O, as flash "
                       "attention's backward forms it (ms_per_step_with_f32_O: the forward also writes a "
                       "float32 O with unrounded P and D comes from it)",
           "ms_per_step_one_stream": {"graph": round(ms_seq, 4), "eager": round(ms_seq_eager, 4)},
           "schedule": "each segment's backward on one of two side streams (even and odd segments) after "
                       "its own forward, beside the next segments' forwards and the previous backward (no "
                       "data dependency between them); launched eagerly",
           "selection_density_16k": round(st.density(), 4),
           "selection_density_last_segment": round(st.density([n_seg - 1]), 4),
           "paper_density_16k": 0.087,
           "phases_16k": phases, "sum_of_calls_ms_per_step": round(eager_ms, 4),
           "segments_16k_us": {k: [round(v[i] * 1e3, 2) for i in range(n_seg)]
                               for k, v in (("summaries", sum_seg), ("route_attend_fwd", fwd_seg),
                                            ("attend_bwd", bwd_seg))},
           "peak_mem_MB_16k": round(peak_mb, 1),
           "fwd_tokens_per_s_16k": round(wl.T / (per_step["summaries"] + per_step["route_attend_fwd"]) * 1e3, 1)}
    gpu_routing = dict(st.routing)
    del st
    torch.cuda.empty_cache()
    # every further configuration in a fresh process (the paper runs each
    # context length in its own subprocess)
    if not args.no_131k:
        sweep = {T: run_part(["--part", "context", "--context-T", str(T), "--event-reps", str(args.event_reps)])
                 for T in CONTEXT_SWEEP}
        out["fwd_131k"] = sweep[131072]
        out["fwd_context_sweep"] = [{"T": T, "ms": r["ms"], "tokens_per_s": r["tokens_per_s"],
                                     "us_per_1k_tokens": r["us_per_1k_tokens"],
                                     "selection_density": r["selection_density"],
                                     "dense_ms": r["dense_fwd"]["ms"],
                                     "dense_TFLOP/s": r["dense_fwd"]["TFLOP/s"],
                                     "hga_speedup_vs_dense": r["dense_fwd"]["hga_speedup"]}
                                    for T, r in sweep.items()]
    if not args.no_sweep:
        out["routing_sweep_32k"] = run_part(["--part", "sweep", "--event-reps", str(args.event_reps)])
    if not args.no_rows:
        out["per_query_routing"] = run_part(["--part", "rows", "--event-reps", str(args.event_reps)])
    if not args.no_dense:
        out["training_vs_dense"] = run_part(["--part", "dense", "--event-reps", str(args.event_reps)])
    if not args.no_tier:
        out["tiered_16k"] = run_part(["--part", "tier", "--event-reps", str(args.event_reps)])
    if not args.no_cpu_baseline:
        log("[bench] CPU oracle baseline")
        out["cpu_baseline"] = cpu_baseline(wl, gpu_routing)
    print(json.dumps(out), flush=True)


CONTEXT_SWEEP = (2048, 8192, 16384, 32768, 65536, 131072)


def run_part(extra):
    """Run `bench.py --part ...` in a child process and return its result
    (the child prints one `part_json:` line)."""
    import subprocess
    cmd = [sys.executable, os.path.abspath(__file__), *extra]
    log(f"[bench] fresh process: {' '.join(extra)}")
    r = subprocess.run(cmd, stdout=subprocess.PIPE, text=True, timeout=900)
    if r.returncode != 0:
        raise RuntimeError(f"bench part {extra} failed with status {r.returncode}")
    for line in r.stdout.splitlines():
        if line.startswith("part_json: "):
            return json.loads(line[len("part_json: "):])
    raise RuntimeError(f"bench part {extra} printed no result")


def main_part(args):
    if args.part == "context":
        wl = synth.WORKLOADS["qwen3_8b_131k_planted"]
        res = bench_forward(dataclasses.replace(wl, T=args.context_T, n_q=args.context_T), args.event_reps)
    elif args.part == "rows":
        res = bench_rows(args.event_reps)
    elif args.part == "dense":
        res = bench_dense_training(args.event_reps)
    elif args.part == "tier":
        res = bench_tier(args.event_reps)
    else:
        res = bench_routing_sweep(args.event_reps)
    print("part_json: " + json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
