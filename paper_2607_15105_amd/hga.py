"""Thin ctypes binding of libhga.so (C ABI in include/hga.h).

Argument marshalling only: torch tensors provide device memory and the current
HIP stream; every step of the hot path runs in the library's HIP kernels.
There is no fallback: if the library is missing, every call raises.

Function names follow the C ABI without the ``hga_`` prefix.
"""

from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libhga.so")
_lib = None

HGA_F32, HGA_BF16 = 0, 1
OP_ROUTE, OP_BWD = 0, 1
NOALLOC_SCRATCH_BYTES = 48 << 20  # HGA_NOALLOC_SCRATCH_BYTES
STATUS = {0: "ok", -1: "invalid argument", -2: "unsupported configuration",
          -3: "workspace missing or too small", -4: "HIP launch or runtime error"}


class HgaError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn} failed: {STATUS.get(status, status)} ({status})")
        self.status = status


class Config(ctypes.Structure):
    """hga_config_t."""
    _fields_ = [("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("chunk_size", ctypes.c_int32),
                ("group_size", ctypes.c_int32), ("query_block", ctypes.c_int32),
                ("top_chunks", ctypes.c_int32), ("top_groups", ctypes.c_int32),
                ("sink_tokens", ctypes.c_int32), ("local_tokens", ctypes.c_int32),
                ("softmax_scale", ctypes.c_float), ("dtype", ctypes.c_int32),
                ("bwd_kv_parts", ctypes.c_int32)]


class GroupCache(ctypes.Structure):
    """hga_group_cache_t: device buffers of a bounded group-summary cache."""
    _fields_ = [("slot_of", ctypes.c_void_p), ("slot_chunk", ctypes.c_void_p), ("cursor", ctypes.c_void_p),
                ("groups", ctypes.c_void_p), ("n_slots", ctypes.c_int64), ("chunk_cap", ctypes.c_int64)]


class Strides(ctypes.Structure):
    """hga_strides_t (element strides; head_dim axis contiguous)."""
    _fields_ = [("token", ctypes.c_int64), ("head", ctypes.c_int64)]


def library_path() -> str:
    return _LIB_PATH


def lib() -> ctypes.CDLL:
    """Load libhga.so once; raise if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is missing: build it with "
                               "`python -m paper_2607_15105_amd.build`")
        L = ctypes.CDLL(_LIB_PATH)
        P, I64, SZ = ctypes.c_void_p, ctypes.c_int64, ctypes.c_size_t
        C, S = ctypes.POINTER(Config), Strides
        L.hga_build_summaries.argtypes = [C, P, S, I64, I64, P, I64, P, I64, P]
        L.hga_route.argtypes = [C, P, S, I64, I64, P, I64, P, I64, P, P, P, P, SZ, P]
        L.hga_attend_fwd.argtypes = [C, P, S, P, S, P, S, I64, I64, P, P, P, S, P, P, P]
        L.hga_route_attend_fwd.argtypes = [C, P, S, P, S, P, S, I64, I64, P, I64, P, I64, P, P, P,
                                           P, S, P, P, P, SZ, P]
        L.hga_attend_bwd.argtypes = [C, P, S, P, S, P, S, P, S, P, P, S, P, I64, I64, I64, P, P,
                                     P, P, P, P, SZ, P]
        L.hga_attend_bwd_noalloc.argtypes = [C, P, S, P, S, P, S, P, S, P, P, S, P, I64, I64, I64, P,
                                             P, P, P, P, P]
        L.hga_route_rows.argtypes = [C, P, S, I64, I64, P, I64, P, I64, P, P, P, P]
        L.hga_attend_rows_fwd.argtypes = [C, P, S, P, S, P, S, I64, I64, P, P, P, S, P, P, P]
        L.hga_attend_rows_bwd.argtypes = [C, P, S, P, S, P, S, P, S, P, P, S, P, I64, I64, I64, P, P,
                                          P, P, P, P, SZ, P]
        L.hga_rows_workspace_size.argtypes = [C, I64]
        L.hga_rows_workspace_size.restype = SZ
        G = ctypes.POINTER(GroupCache)
        L.hga_host_device_view.argtypes = [P]
        L.hga_host_device_view.restype = P
        L.hga_group_cache_clear.argtypes = [C, G, P]
        L.hga_route_cached.argtypes = [C, P, S, I64, I64, P, I64, P, I64, G, P, P, P, P, P, SZ, P]
        L.hga_group_cache_update.argtypes = [C, G, P, I64, I64, I64, P, P, P]
        L.hga_gather_tiered.argtypes = [C, P, P, S, I64, P, P, S, I64, I64, P, P, P, P, I64, P]
        L.hga_attend_gathered_bwd.argtypes = [C, P, S, P, P, I64, P, P, S, I64, P, S, P, P, S, P, I64, I64, I64,
                                              P, P, P, P, P, P, SZ, P]
        L.hga_gather_routed.argtypes = [C, P, S, P, S, I64, I64, P, P, P, P, I64, P]
        L.hga_attend_gathered_fwd.argtypes = [C, P, S, P, P, I64, I64, I64, P, P, S, P, P, P]
        L.hga_workspace_size.argtypes = [C, ctypes.c_int, I64, I64, I64]
        L.hga_workspace_size.restype = SZ
        L.hga_status_string.argtypes = [ctypes.c_int]
        L.hga_status_string.restype = ctypes.c_char_p
        for fn in ("hga_build_summaries", "hga_route", "hga_attend_fwd", "hga_route_attend_fwd",
                   "hga_attend_bwd", "hga_attend_bwd_noalloc", "hga_gather_routed",
                   "hga_attend_gathered_fwd", "hga_route_rows", "hga_attend_rows_fwd",
                   "hga_attend_rows_bwd", "hga_group_cache_clear", "hga_route_cached",
                   "hga_group_cache_update", "hga_gather_tiered", "hga_attend_gathered_bwd"):
            getattr(L, fn).restype = ctypes.c_int
        _lib = L
    return _lib


def make_config(n_q_heads: int, n_kv_heads: int, head_dim: int, *, chunk_size: int = 64,
                group_size: int = 8, query_block: int = 64, top_chunks: int = 8,
                top_groups: int = 16, sink_tokens: int = 64, local_tokens: int = 128,
                softmax_scale: float = 0.0, dtype=torch.bfloat16, bwd_kv_parts: int = 0) -> Config:
    if dtype not in (torch.bfloat16, torch.float32):
        raise ValueError("dtype must be torch.bfloat16 or torch.float32")
    return Config(n_q_heads, n_kv_heads, head_dim, chunk_size, group_size, query_block,
                  top_chunks, top_groups, sink_tokens, local_tokens, softmax_scale,
                  HGA_BF16 if dtype == torch.bfloat16 else HGA_F32, bwd_kv_parts)


def _ptr(t: torch.Tensor | None) -> int | None:
    return None if t is None else t.data_ptr()


def _strides(t: torch.Tensor) -> Strides:
    if t.dim() != 3 or t.stride(2) != 1:
        raise ValueError("expected a [rows, heads, head_dim] tensor with contiguous head_dim")
    return Strides(t.stride(0), t.stride(1))


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def _check(fn: str, status: int) -> None:
    if status != 0:
        raise HgaError(fn, status)


_recording: list | None = None


def _call(fn: str, *args) -> None:
    """Make ABI call `fn` with marshalled `args`, or, inside `record()`, keep
    it for later."""
    if _recording is not None:
        _recording.append(PreparedCall(fn, args))
        return
    _check(fn, getattr(lib(), fn)(*args))


class PreparedCall:
    """One ABI call with its arguments marshalled once: device addresses,
    strides, sizes and the HIP stream current when it was recorded. Calling
    it issues the same call again with no other host work, for launch loops
    such as a training step. The tensors it was recorded from must stay
    alive and in place."""

    __slots__ = ("name", "fn", "args")

    def __init__(self, name: str, args: tuple):
        self.name = name
        self.fn = getattr(lib(), name)
        # numbers as ctypes values of the parameter types, built once
        self.args = tuple(t(a) if isinstance(a, (int, float)) and issubclass(t, ctypes._SimpleCData) else a
                          for t, a in zip(self.fn.argtypes, args))

    def __call__(self) -> None:
        status = self.fn(*self.args)
        if status != 0:
            raise HgaError(self.name, status)


class record:
    """Context manager: the ABI calls made inside it are not issued but kept,
    as PreparedCall objects, in the list it returns."""

    def __enter__(self) -> list:
        global _recording
        if _recording is not None:
            raise RuntimeError("hga.record() does not nest")
        _recording = []
        return _recording

    def __exit__(self, *exc) -> None:
        global _recording
        _recording = None


def workspace_size(cfg: Config, op: int, q_begin: int, n_q: int, grad_begin: int | None = None) -> int:
    """Workspace bytes; grad_begin (backward only) defaults to q_begin."""
    gb = q_begin if grad_begin is None else grad_begin
    return int(lib().hga_workspace_size(ctypes.byref(cfg), op, q_begin, n_q, gb))


def build_summaries(cfg: Config, K: torch.Tensor, t_begin: int, t_end: int,
                    chunk_sum: torch.Tensor, group_sum: torch.Tensor) -> None:
    """Summaries of tokens [t_begin, t_end) into the quad-major tables
    chunk_sum[Hkv, d/4, cap, 4] and group_sum[Hkv, d/4, cap, 4]."""
    _call("hga_build_summaries",
        ctypes.byref(cfg), _ptr(K), _strides(K), t_begin, t_end, _ptr(chunk_sum),
        chunk_sum.shape[2], _ptr(group_sum), group_sum.shape[2], _stream())


def build_summaries_raw(cfg: Config, k_ptr: int, k_strides: Strides, t_begin: int, t_end: int,
                        chunk_sum: torch.Tensor, group_sum, group_cap: int) -> None:
    """build_summaries with K and the group table given as addresses (a
    shifted device view, or the device view of a host table)."""
    _call("hga_build_summaries",
        ctypes.byref(cfg), k_ptr, k_strides, t_begin, t_end, _ptr(chunk_sum), chunk_sum.shape[2],
        _pp(group_sum), group_cap, _stream())


def route(cfg: Config, Q: torch.Tensor, q_begin: int, chunk_sum: torch.Tensor,
          group_sum: torch.Tensor, sel_chunks: torch.Tensor, sel_groups: torch.Tensor,
          n_sel_groups: torch.Tensor, workspace: torch.Tensor) -> None:
    n_q = Q.shape[0]
    _call("hga_route",
        ctypes.byref(cfg), _ptr(Q), _strides(Q), q_begin, n_q, _ptr(chunk_sum),
        chunk_sum.shape[2], _ptr(group_sum), group_sum.shape[2], _ptr(sel_chunks),
        _ptr(sel_groups), _ptr(n_sel_groups), _ptr(workspace), workspace.numel(), _stream())


def attend_fwd(cfg: Config, Q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, q_begin: int,
               sel_groups: torch.Tensor, n_sel_groups: torch.Tensor, O: torch.Tensor,
               lse: torch.Tensor, o_f32: torch.Tensor | None = None) -> None:
    _call("hga_attend_fwd",
        ctypes.byref(cfg), _ptr(Q), _strides(Q), _ptr(K), _strides(K), _ptr(V), _strides(V),
        q_begin, Q.shape[0], _ptr(sel_groups), _ptr(n_sel_groups), _ptr(O), _strides(O),
        _ptr(lse), _ptr(o_f32), _stream())


def route_attend_fwd(cfg: Config, Q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, q_begin: int,
                     chunk_sum: torch.Tensor, group_sum: torch.Tensor, sel_chunks: torch.Tensor,
                     sel_groups: torch.Tensor, n_sel_groups: torch.Tensor, O: torch.Tensor,
                     lse: torch.Tensor, workspace: torch.Tensor, o_f32: torch.Tensor | None = None) -> None:
    """route() then attend_fwd() on the same rows (one launch for segment-sized calls)."""
    _call("hga_route_attend_fwd",
        ctypes.byref(cfg), _ptr(Q), _strides(Q), _ptr(K), _strides(K), _ptr(V), _strides(V),
        q_begin, Q.shape[0], _ptr(chunk_sum), chunk_sum.shape[2], _ptr(group_sum), group_sum.shape[2],
        _ptr(sel_chunks), _ptr(sel_groups), _ptr(n_sel_groups), _ptr(O), _strides(O), _ptr(lse),
        _ptr(o_f32), _ptr(workspace), workspace.numel(), _stream())


def attend_bwd(cfg: Config, Q, K, V, O, dO, lse, q_begin: int, grad_begin: int, sel_groups,
               n_sel_groups, dQ, dK, dV, workspace: torch.Tensor,
               o_f32: torch.Tensor | None = None) -> None:
    _call("hga_attend_bwd",
        ctypes.byref(cfg), _ptr(Q), _strides(Q), _ptr(K), _strides(K), _ptr(V), _strides(V),
        _ptr(O), _strides(O), _ptr(o_f32), _ptr(dO), _strides(dO), _ptr(lse), q_begin,
        Q.shape[0], grad_begin, _ptr(sel_groups), _ptr(n_sel_groups), _ptr(dQ), _ptr(dK),
        _ptr(dV), _ptr(workspace), workspace.numel(), _stream())


def attend_bwd_noalloc(cfg: Config, Q, K, V, O, dO, lse, q_begin: int, grad_begin: int, sel_groups,
                       n_sel_groups, dQ, dK, dV, o_f32: torch.Tensor | None = None) -> None:
    """attend_bwd with the library's static scratch instead of a workspace
    (for callers that cannot allocate)."""
    _call("hga_attend_bwd_noalloc",
        ctypes.byref(cfg), _ptr(Q), _strides(Q), _ptr(K), _strides(K), _ptr(V), _strides(V),
        _ptr(O), _strides(O), _ptr(o_f32), _ptr(dO), _strides(dO), _ptr(lse), q_begin,
        Q.shape[0], grad_begin, _ptr(sel_groups), _ptr(n_sel_groups), _ptr(dQ), _ptr(dK),
        _ptr(dV), _stream())


def route_rows(cfg: Config, Q: torch.Tensor, q_begin: int, chunk_sum: torch.Tensor,
               group_sum: torch.Tensor, sel_chunks: torch.Tensor, sel_groups: torch.Tensor,
               n_sel_groups: torch.Tensor) -> None:
    """Per-query routing of the rows of Q (row i at position q_begin + i)."""
    _call("hga_route_rows",
        ctypes.byref(cfg), _ptr(Q), _strides(Q), q_begin, Q.shape[0], _ptr(chunk_sum),
        chunk_sum.shape[2], _ptr(group_sum), group_sum.shape[2], _ptr(sel_chunks),
        _ptr(sel_groups), _ptr(n_sel_groups), _stream())


def attend_rows_fwd(cfg: Config, Q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, q_begin: int,
                    sel_groups: torch.Tensor, n_sel_groups: torch.Tensor, O: torch.Tensor,
                    lse: torch.Tensor, o_f32: torch.Tensor | None = None) -> None:
    """Attention of each row of Q over its own routed set (from route_rows)."""
    _call("hga_attend_rows_fwd",
        ctypes.byref(cfg), _ptr(Q), _strides(Q), _ptr(K), _strides(K), _ptr(V), _strides(V),
        q_begin, Q.shape[0], _ptr(sel_groups), _ptr(n_sel_groups), _ptr(O), _strides(O),
        _ptr(lse), _ptr(o_f32), _stream())


def rows_workspace_size(cfg: Config, n_q: int) -> int:
    return int(lib().hga_rows_workspace_size(ctypes.byref(cfg), n_q))


def attend_rows_bwd(cfg: Config, Q, K, V, O, dO, lse, q_begin: int, grad_begin: int, sel_groups,
                    n_sel_groups, dQ, dK, dV, workspace: torch.Tensor,
                    o_f32: torch.Tensor | None = None) -> None:
    """Backward of attend_rows_fwd (dK/dV for tokens >= grad_begin)."""
    _call("hga_attend_rows_bwd",
        ctypes.byref(cfg), _ptr(Q), _strides(Q), _ptr(K), _strides(K), _ptr(V), _strides(V),
        _ptr(O), _strides(O), _ptr(o_f32), _ptr(dO), _strides(dO), _ptr(lse), q_begin,
        Q.shape[0], grad_begin, _ptr(sel_groups), _ptr(n_sel_groups), _ptr(dQ), _ptr(dK),
        _ptr(dV), _ptr(workspace), workspace.numel(), _stream())


def alloc_route_rows(cfg: Config, n_q: int, device="cuda"):
    """(sel_chunks, sel_groups, n_sel_groups) for n_q rows of per-query routing."""
    return (torch.empty(n_q, cfg.n_kv_heads, max(cfg.top_chunks, 1), dtype=torch.int32, device=device),
            torch.empty(n_q, cfg.n_kv_heads, max(cfg.top_groups, 1), dtype=torch.int32, device=device),
            torch.empty(n_q, cfg.n_kv_heads, dtype=torch.int32, device=device))


def gather_routed(cfg: Config, K: torch.Tensor, V: torch.Tensor, q_begin: int, n_q: int,
                  sel_groups: torch.Tensor, n_sel_groups: torch.Tensor, Kc: torch.Tensor,
                  Vc: torch.Tensor) -> None:
    """Routed K/V rows of every (block, kv head) into Kc, Vc [n_q/B, Hkv, r_cap, d]."""
    if Kc.shape != Vc.shape or Kc.dim() != 4 or not (Kc.is_contiguous() and Vc.is_contiguous()):
        raise ValueError("Kc, Vc: dense [n_q/B, Hkv, r_cap, d] tensors of one shape")
    _call("hga_gather_routed",
        ctypes.byref(cfg), _ptr(K), _strides(K), _ptr(V), _strides(V), q_begin, n_q,
        _ptr(sel_groups), _ptr(n_sel_groups), _ptr(Kc), _ptr(Vc), Kc.shape[2], _stream())


def attend_gathered_fwd(cfg: Config, Q: torch.Tensor, Kc: torch.Tensor, Vc: torch.Tensor,
                        q_begin: int, n_sel_groups: torch.Tensor, O: torch.Tensor,
                        lse: torch.Tensor, o_f32: torch.Tensor | None = None) -> None:
    """attend_fwd over the compact rows written by gather_routed."""
    if Kc.shape != Vc.shape or Kc.dim() != 4 or not (Kc.is_contiguous() and Vc.is_contiguous()):
        raise ValueError("Kc, Vc: dense [n_q/B, Hkv, r_cap, d] tensors of one shape")
    _call("hga_attend_gathered_fwd",
        ctypes.byref(cfg), _ptr(Q), _strides(Q), _ptr(Kc), _ptr(Vc), Kc.shape[2], q_begin,
        Q.shape[0], _ptr(n_sel_groups), _ptr(O), _strides(O), _ptr(lse), _ptr(o_f32), _stream())


def gathered_rows(cfg: Config) -> int:
    """Smallest r_cap (rows per slot) that hga_gather_routed accepts."""
    r = cfg.sink_tokens + cfg.local_tokens + cfg.top_groups * cfg.group_size
    return -(-r // 64) * 64


# ---------------------------------------------------------------------------
# Tiered storage: host-RAM history and a bounded group-summary cache
# ---------------------------------------------------------------------------

def host_view(t: torch.Tensor) -> int:
    """Device-mapped address of a pinned host tensor (raises if not pinned)."""
    if t.device.type != "cpu" or not t.is_pinned():
        raise ValueError("expected a pinned host tensor")
    p = lib().hga_host_device_view(t.data_ptr())
    if not p:
        raise HgaError("hga_host_device_view", -1)
    return int(p)


def shifted_rows(t: torch.Tensor, first_token: int) -> int:
    """Address token 0 would have in a token-major tensor whose row 0 is token
    `first_token`: entry points index K by absolute token, and only rows from
    first_token on are read."""
    return t.data_ptr() - first_token * t.stride(0) * t.element_size()


@dataclass
class Cache:
    """Device buffers of a group-summary cache and their descriptor."""
    slot_of: torch.Tensor
    slot_chunk: torch.Tensor
    cursor: torch.Tensor
    groups: torch.Tensor
    desc: GroupCache


def alloc_group_cache(cfg: Config, n_slots: int, chunk_cap: int, device="cuda") -> Cache:
    gpc = cfg.chunk_size // cfg.group_size
    so = torch.empty(cfg.n_kv_heads, chunk_cap, dtype=torch.int32, device=device)
    sc = torch.empty(cfg.n_kv_heads, n_slots, dtype=torch.int32, device=device)
    cu = torch.empty(cfg.n_kv_heads, dtype=torch.int32, device=device)
    gr = torch.empty(cfg.n_kv_heads, cfg.head_dim // 4, n_slots * gpc, 4, device=device)
    return Cache(so, sc, cu, gr, GroupCache(so.data_ptr(), sc.data_ptr(), cu.data_ptr(), gr.data_ptr(),
                                            n_slots, chunk_cap))


def group_cache_clear(cfg: Config, cache: Cache) -> None:
    _call("hga_group_cache_clear", ctypes.byref(cfg), ctypes.byref(cache.desc), _stream())


def _pp(x) -> int | None:
    """Pointer of a tensor, or an address given as an int."""
    return x if isinstance(x, int) or x is None else x.data_ptr()


def route_cached(cfg: Config, Q: torch.Tensor, q_begin: int, chunk_sum: torch.Tensor, group_sum,
                 group_cap: int, cache: Cache, sel_chunks, sel_groups, n_sel_groups, cache_hit,
                 workspace: torch.Tensor) -> None:
    """Routing with group summaries from the cache where resident, else from
    group_sum (a tensor or the device view of a host table, group_cap rows)."""
    _call("hga_route_cached",
        ctypes.byref(cfg), _ptr(Q), _strides(Q), q_begin, Q.shape[0], _ptr(chunk_sum), chunk_sum.shape[2],
        _pp(group_sum), group_cap, ctypes.byref(cache.desc), _ptr(sel_chunks), _ptr(sel_groups),
        _ptr(n_sel_groups), _ptr(cache_hit), _ptr(workspace), workspace.numel(), _stream())


def group_cache_update(cfg: Config, cache: Cache, group_sum, group_cap: int, q_begin: int, n_q: int,
                       sel_chunks, cache_hit) -> None:
    _call("hga_group_cache_update",
        ctypes.byref(cfg), ctypes.byref(cache.desc), _pp(group_sum), group_cap, q_begin, n_q, _ptr(sel_chunks),
        _ptr(cache_hit), _stream())


def gather_tiered(cfg: Config, K_hist, V_hist, hist_strides: Strides, hist_end: int, K_act: torch.Tensor,
                  V_act: torch.Tensor, q_begin: int, n_q: int, sel_groups, n_sel_groups, Kc: torch.Tensor,
                  Vc: torch.Tensor) -> None:
    """Routed rows into Kc, Vc: tokens < hist_end from K_hist / V_hist
    (device views of host tensors, or tensors), the others from K_act / V_act
    (row 0 = token hist_end)."""
    _call("hga_gather_tiered",
        ctypes.byref(cfg), _pp(K_hist), _pp(V_hist), hist_strides, hist_end, _ptr(K_act), _ptr(V_act),
        _strides(K_act), q_begin, n_q, _ptr(sel_groups), _ptr(n_sel_groups), _ptr(Kc), _ptr(Vc), Kc.shape[2],
        _stream())


def attend_gathered_bwd(cfg: Config, Q, Kc, Vc, K_act, V_act, act_begin: int, O, dO, lse, q_begin: int,
                        grad_begin: int, sel_groups, n_sel_groups, dQ, dK, dV, workspace: torch.Tensor,
                        o_f32: torch.Tensor | None = None) -> None:
    """The backward over compact routed rows; dK/dV keys from K_act / V_act
    (row 0 = token act_begin)."""
    _call("hga_attend_gathered_bwd",
        ctypes.byref(cfg), _ptr(Q), _strides(Q), _ptr(Kc), _ptr(Vc), Kc.shape[2], _ptr(K_act), _ptr(V_act),
        _strides(K_act), act_begin, _ptr(O), _strides(O), _ptr(o_f32), _ptr(dO), _strides(dO), _ptr(lse),
        q_begin, Q.shape[0], grad_begin, _ptr(sel_groups), _ptr(n_sel_groups), _ptr(dQ), _ptr(dK), _ptr(dV),
        _ptr(workspace), workspace.numel(), _stream())


# ---------------------------------------------------------------------------
# Convenience: torch-owned buffers sized for one call (allocation stays with
# the caller, as the C ABI requires).
# ---------------------------------------------------------------------------

@dataclass
class RouteBuffers:
    sel_chunks: torch.Tensor
    sel_groups: torch.Tensor
    n_sel_groups: torch.Tensor
    workspace: torch.Tensor


def alloc_summaries(cfg: Config, T: int, device="cuda"):
    """Chunk and group summary tables for T tokens, quad-major [Hkv, d/4, cap, 4]."""
    d = cfg.head_dim
    return (torch.zeros(cfg.n_kv_heads, d // 4, T // cfg.chunk_size, 4, device=device),
            torch.zeros(cfg.n_kv_heads, d // 4, T // cfg.group_size, 4, device=device))


def summary_rows(table: torch.Tensor) -> torch.Tensor:
    """A quad-major summary table as rows [Hkv, cap, d] (a copy)."""
    h, q, cap, _ = table.shape
    return table.permute(0, 2, 1, 3).reshape(h, cap, 4 * q)


def alloc_route(cfg: Config, q_begin: int, n_q: int, device="cuda") -> RouteBuffers:
    n_qb = n_q // cfg.query_block
    return RouteBuffers(
        torch.empty(n_qb, cfg.n_kv_heads, max(cfg.top_chunks, 1), dtype=torch.int32, device=device),
        torch.empty(n_qb, cfg.n_kv_heads, max(cfg.top_groups, 1), dtype=torch.int32, device=device),
        torch.empty(n_qb, cfg.n_kv_heads, dtype=torch.int32, device=device),
        torch.empty(max(workspace_size(cfg, OP_ROUTE, q_begin, n_q), 256), dtype=torch.uint8,
                    device=device))
