"""Seeded synthetic inputs for the HGA hot path.

This module only draws random tensors with the shapes and structure of the
workloads; it holds none of the method's arithmetic, so both the CPU oracle
and the GPU library can be fed from it.

Stand-ins: the paper trains and evaluates Qwen3-8B on PG19 text (Sec. 3) and
probes retrieval with a RULER-style suite (Sec. 4.6). Neither the weights nor
the data are available, so every tensor here is synthetic with Qwen3-8B layer
shapes (32 query heads, 8 kv heads, head dim 128, GQA 4:1) and a structure
that makes routing non-degenerate (per-chunk key offsets) or checkable
(planted key groups aligned to probe queries).

Every tensor is produced in slabs of ``SLAB`` tokens, each drawn from a
PCG64 stream keyed by (seed, tensor id, slab), so any token range can be
regenerated on its own. Floating values are drawn as float32; bf16 tensors are
rounded to nearest-even and returned as uint16 bit patterns.
"""

from __future__ import annotations

import concurrent.futures as cf
import math
import os
from dataclasses import dataclass, replace

import numpy as np

SLAB = 2048
_WORKERS = min(16, os.cpu_count() or 1)


def _map_slabs(fn, slabs):
    """fn over slab ids on a thread pool (each slab has its own stream: same result)."""
    slabs = list(slabs)
    if len(slabs) <= 1:
        return [fn(s) for s in slabs]
    with cf.ThreadPoolExecutor(max_workers=_WORKERS) as ex:
        return list(ex.map(fn, slabs))

_K, _V, _Q, _DO, _OFFSET, _PLANT, _PLANT_W, _PROBE, _TIE = range(1, 10)


@dataclass(frozen=True)
class Workload:
    name: str
    T: int                      # tokens of context
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    dtype: str                  # "fp32" or "bf16"
    seed: int
    q_begin: int                # first query row of the (last) call
    n_q: int                    # query rows of one call
    grad_begin: int             # first token with dK/dV
    segment: int = 0            # > 0: the context is processed as T/segment calls
    key_offset: str = "none"    # "none" | "normal" | "student_t"
    offset_scale: float = 0.5
    planted: bool = False
    tie_copies: int = 0
    backward: bool = True
    chunk_size: int = 64
    group_size: int = 8
    query_block: int = 64
    top_chunks: int = 8
    top_groups: int = 16
    sink_tokens: int = 64
    local_tokens: int = 128

    def with_budget(self, **kw) -> "Workload":
        return replace(self, **kw)


WORKLOADS = {
    # 1 head, head dim 64, 1,024 tokens, float32, forward only.
    "tiny_fp32_1k": Workload("tiny_fp32_1k", T=1024, n_q_heads=1, n_kv_heads=1, head_dim=64,
                             dtype="fp32", seed=0, q_begin=0, n_q=1024, grad_begin=0,
                             top_chunks=4, top_groups=8, sink_tokens=64, local_tokens=64,
                             backward=False),
    # Qwen3-8B layer shape, one 2,048-token segment, forward + backward.
    "qwen3_8b_2k": Workload("qwen3_8b_2k", T=2048, n_q_heads=32, n_kv_heads=8, head_dim=128,
                            dtype="bf16", seed=2, q_begin=0, n_q=2048, grad_begin=0,
                            key_offset="normal"),
    # 16,384 tokens as sixteen 1,024-token segments; only the current one is differentiable.
    "qwen3_8b_16k_seg1k": Workload("qwen3_8b_16k_seg1k", T=16384, n_q_heads=32, n_kv_heads=8,
                                   head_dim=128, dtype="bf16", seed=3, q_begin=15360, n_q=1024,
                                   grad_begin=15360, segment=1024, key_offset="normal"),
    # 131,072-token forward with 64 planted groups aligned to the last 8 query blocks.
    "qwen3_8b_131k_planted": Workload("qwen3_8b_131k_planted", T=131072, n_q_heads=32,
                                      n_kv_heads=8, head_dim=128, dtype="bf16", seed=4,
                                      q_begin=0, n_q=131072, grad_begin=0, key_offset="normal",
                                      planted=True, backward=False, top_chunks=16,
                                      top_groups=32, local_tokens=256),
    # 32,768 tokens, backward over the last 2,048; heavy-tailed chunk offsets.
    "qwen3_8b_32k_sweep": Workload("qwen3_8b_32k_sweep", T=32768, n_q_heads=32, n_kv_heads=8,
                                   head_dim=128, dtype="bf16", seed=5, q_begin=30720, n_q=2048,
                                   grad_begin=30720, key_offset="student_t"),
}

# The routing sweep of the 32K workload: group size x top chunks x top groups.
SWEEP = [(g, kc, kg) for g in (8, 16) for kc in (4, 8, 16, 32) for kg in (8, 32, 64)]

N_PLANTED_CHUNKS = 16
PLANTED_GROUPS_PER_CHUNK = 4
N_PROBE_BLOCKS = 8
PLANT_COS = 0.9


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (nearest, ties to even); returns uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> 16) & 1) + np.uint32(0x7FFF)
    return ((u + bias) >> 16).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _rng(*key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(list(key))))


def _cast(wl: Workload, x: np.ndarray) -> np.ndarray:
    return to_bf16_bits(x) if wl.dtype == "bf16" else x.astype(np.float32)


def _unit(x: np.ndarray) -> np.ndarray:
    return x / np.linalg.norm(x, axis=-1, keepdims=True)


def _orthogonal_unit(rng, u: np.ndarray, n: int) -> np.ndarray:
    """n random unit vectors orthogonal to the unit vector u."""
    z = rng.standard_normal((n, u.shape[0]))
    z -= (z @ u)[:, None] * u[None, :]
    return _unit(z)


def chunk_offsets(wl: Workload) -> np.ndarray:
    """Per-(chunk, kv head) key offset vectors, float32 [T/C, Hkv, d]."""
    shape = (wl.T // wl.chunk_size, wl.n_kv_heads, wl.head_dim)
    rng = _rng(wl.seed, _OFFSET)
    if wl.key_offset == "normal":
        return (wl.offset_scale * rng.standard_normal(shape)).astype(np.float32)
    if wl.key_offset == "student_t":
        return (wl.offset_scale * rng.standard_t(3.0, shape)).astype(np.float32)
    return np.zeros(shape, np.float32)


@dataclass(frozen=True)
class Plant:
    directions: np.ndarray      # [Hkv, d] unit vectors u_h
    chunks: np.ndarray          # [16] planted chunk ids (ascending)
    groups: np.ndarray          # [16, 4] planted group ids (global)
    probe_blocks: np.ndarray    # absolute query block ids whose queries probe u_h


def plant(wl: Workload) -> Plant:
    """Where the planted groups sit: 16 chunks spread evenly over tokens [64, T/2)."""
    rng = _rng(wl.seed, _PLANT)
    C, g = wl.chunk_size, wl.group_size
    u = _unit(rng.standard_normal((wl.n_kv_heads, wl.head_dim)))
    first, last = 1, (wl.T // 2) // C
    chunks = first + (np.arange(N_PLANTED_CHUNKS) * (last - first)) // N_PLANTED_CHUNKS
    groups = np.stack([c * (C // g) + np.sort(rng.choice(C // g, PLANTED_GROUPS_PER_CHUNK,
                                                         replace=False)) for c in chunks])
    n_blocks = wl.T // wl.query_block
    probes = np.arange(n_blocks - N_PROBE_BLOCKS, n_blocks)
    return Plant(u, chunks.astype(np.int64), groups.astype(np.int64), probes)


def _tie_pairs(wl: Workload):
    """(dst, src) chunk pairs: dst's keys become a bit-identical copy of src's."""
    if wl.tie_copies == 0:
        return []
    rng = _rng(wl.seed, _TIE)
    n = wl.T // wl.chunk_size
    picks = rng.choice(np.arange(1, n - 8), 2 * wl.tie_copies, replace=False)
    return [(int(picks[2 * i]), int(picks[2 * i + 1])) for i in range(wl.tie_copies)]


def _key_slab(wl: Workload, s: int, offsets: np.ndarray, pl: Plant | None) -> np.ndarray:
    C, g = wl.chunk_size, wl.group_size
    n = min(SLAB, wl.T - s * SLAB)
    k = _rng(wl.seed, _K, s).standard_normal((SLAB, wl.n_kv_heads, wl.head_dim),
                                             dtype=np.float32)[:n]
    t0 = s * SLAB
    k += offsets[(t0 + np.arange(n)) // C]
    if pl is not None:
        for grp in pl.groups.reshape(-1):
            a = grp * g - t0
            if 0 <= a < n:
                rng = _rng(wl.seed, _PLANT_W, int(grp))
                for h in range(wl.n_kv_heads):
                    rows = k[a:a + g, h, :].astype(np.float64)
                    norms = np.linalg.norm(rows, axis=1, keepdims=True)
                    w = _orthogonal_unit(rng, pl.directions[h], g)
                    side = math.sqrt(1.0 - PLANT_COS ** 2)
                    k[a:a + g, h, :] = norms * (PLANT_COS * pl.directions[h][None, :] + side * w)
    return k


def keys(wl: Workload, t0: int = 0, t1: int | None = None) -> np.ndarray:
    """K[t0:t1] as [tokens, Hkv, d] (uint16 bf16 bits or float32)."""
    t1 = wl.T if t1 is None else t1
    offsets = chunk_offsets(wl)
    pl = plant(wl) if wl.planted else None
    pairs = _tie_pairs(wl)
    if pairs:  # copies may cross slabs: build the whole tensor
        full = np.concatenate(_map_slabs(lambda s: _cast(wl, _key_slab(wl, s, offsets, pl)),
                                         range(-(-wl.T // SLAB))))
        C = wl.chunk_size
        for dst, src in pairs:
            full[dst * C:(dst + 1) * C] = full[src * C:(src + 1) * C]
        return full[t0:t1]
    out = _map_slabs(lambda s: _cast(wl, _key_slab(wl, s, offsets, pl)),
                     range(t0 // SLAB, -(-t1 // SLAB)))
    base = (t0 // SLAB) * SLAB
    return np.concatenate(out)[t0 - base:t1 - base]


def _plain(wl: Workload, tid: int, heads: int, t0: int, t1: int, probe: bool = False):
    pl = plant(wl) if (probe and wl.planted) else None

    def one(s):
        n = min(SLAB, wl.T - s * SLAB)
        x = _rng(wl.seed, tid, s).standard_normal((SLAB, heads, wl.head_dim), dtype=np.float32)[:n]
        if pl is not None:
            B = wl.query_block
            G = wl.n_q_heads // wl.n_kv_heads
            rng = _rng(wl.seed, _PROBE, s)
            for blk in pl.probe_blocks:
                a = blk * B - s * SLAB
                if 0 <= a < n:
                    for hq in range(heads):
                        u = pl.directions[hq // G]
                        w = _orthogonal_unit(rng, u, B)
                        side = math.sqrt(1.0 - PLANT_COS ** 2)
                        x[a:a + B, hq, :] = math.sqrt(wl.head_dim) * (PLANT_COS * u[None, :] + side * w)
        return _cast(wl, x)

    out = _map_slabs(one, range(t0 // SLAB, -(-t1 // SLAB)))
    base = (t0 // SLAB) * SLAB
    return np.concatenate(out)[t0 - base:t1 - base]


def values(wl: Workload, t0: int = 0, t1: int | None = None) -> np.ndarray:
    return _plain(wl, _V, wl.n_kv_heads, t0, wl.T if t1 is None else t1)


def queries(wl: Workload, t0: int = 0, t1: int | None = None) -> np.ndarray:
    """Q for absolute token positions [t0, t1) as [rows, Hq, d]."""
    return _plain(wl, _Q, wl.n_q_heads, t0, wl.T if t1 is None else t1, probe=True)


def grad_output(wl: Workload, t0: int = 0, t1: int | None = None) -> np.ndarray:
    """Upstream gradient dO for absolute positions [t0, t1) as [rows, Hq, d]."""
    return _plain(wl, _DO, wl.n_q_heads, t0, wl.T if t1 is None else t1)
