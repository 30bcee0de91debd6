"""SANTA++ decode-time attention for AMD Instinct MI355X (gfx950).

Thin Python binding of libsantapp.so: it marshals torch device tensors into
the C ABI (include/santapp.h) and allocates workspaces; every step of the
method runs in the library's HIP kernels.  There is no CPU fallback: without
the built library every call raises.
"""
from __future__ import annotations

import ctypes
from typing import Optional

import torch

from . import _lib
from ._lib import SantappError, check  # noqa: F401

__all__ = ["Teams", "build_teams", "decode", "decode_static", "dense_decode", "decode_workspace",
           "dense_workspace", "budget_to_K", "SantappError"]


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return _lib.BF16
    if t.dtype == torch.float32:
        return _lib.FP32
    raise SantappError(_lib.EDTYPE, f"unsupported K/V dtype {t.dtype}")


def _ptr(t: Optional[torch.Tensor]):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _need(t: torch.Tensor, name: str, shape=None, dtype=None):
    if not t.is_cuda:
        raise SantappError(_lib.EINVAL, f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise SantappError(_lib.EINVAL, f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise SantappError(_lib.EINVAL, f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if dtype is not None and t.dtype != dtype:
        raise SantappError(_lib.EINVAL, f"{name} has dtype {t.dtype}, expected {dtype}")


class Teams:
    """A team table built by ``santapp_build_teams`` (owns device memory)."""

    def __init__(self, handle: ctypes.c_void_p, torch_dtype):
        self._h = handle
        self.torch_dtype = torch_dtype
        desc = _lib.TeamsDesc()
        check(_lib.load().santapp_teams_info(self._h, ctypes.byref(desc)))
        self.desc = desc
        self.B, self.Hkv, self.N, self.d = desc.B, desc.Hkv, desc.N, desc.d
        self.P, self.R, self.M = desc.parent_size, desc.reps_per_parent, desc.M

    @property
    def handle(self):
        return self._h

    def _view(self, ptr: int, shape, dtype) -> torch.Tensor:
        """Copy a table array into a new tensor (for tests and inspection)."""
        out = torch.empty(shape, dtype=dtype, device="cuda")
        torch.cuda.synchronize()
        _copy_device(out.data_ptr(), ptr, out.numel() * out.element_size())
        return out

    def team_begin(self) -> torch.Tensor:
        return self._view(self.desc.team_begin, (self.B, self.Hkv, self.M), torch.int32)

    def team_size(self) -> torch.Tensor:
        return self._view(self.desc.team_size, (self.B, self.Hkv, self.M), torch.int32)

    def rep_token(self) -> torch.Tensor:
        return self._view(self.desc.rep_token, (self.B, self.Hkv, self.M), torch.int32)

    def perm(self) -> torch.Tensor:
        return self._view(self.desc.perm, (self.B, self.Hkv, self.N), torch.int32)

    def team_count(self) -> torch.Tensor:
        return self._view(self.desc.team_count, (self.B, self.Hkv), torch.int32)

    def packed_K(self) -> torch.Tensor:
        return self._view(self.desc.packed_K, (self.B, self.Hkv, self.N, self.d), self.torch_dtype)

    def packed_V(self) -> torch.Tensor:
        return self._view(self.desc.packed_V, (self.B, self.Hkv, self.N, self.d), self.torch_dtype)

    def reps(self) -> torch.Tensor:
        return self._view(self.desc.reps, (self.B, self.Hkv, self.M, self.d), self.torch_dtype)

    def close(self):
        if self._h is not None and self._h.value:
            _lib.load().santapp_teams_destroy(self._h)
        self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _copy_device(dst: int, src: int, nbytes: int) -> None:
    """Synchronous device-to-device copy through the HIP runtime the library
    itself is linked against."""
    L = _lib.load()
    fn = L.hipMemcpy
    fn.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
    fn.restype = ctypes.c_int
    rc = fn(ctypes.c_void_p(dst), ctypes.c_void_p(src), nbytes, 3)  # device to device
    if rc != 0:
        raise SantappError(_lib.EHIP, f"hipMemcpy failed ({rc})")


def build_teams(K: torch.Tensor, V: torch.Tensor, parent_size: int, reps_per_parent: int,
                stream=None) -> Teams:
    """Team table from prompt K, V ``[B, Hkv, N, d]`` (bf16 or fp32, on the GPU)."""
    _need(K, "K")
    _need(V, "V", shape=K.shape, dtype=K.dtype)
    B, Hkv, N, d = K.shape
    h = ctypes.c_void_p()
    check(_lib.load().santapp_build_teams(_ptr(K), _ptr(V), B, Hkv, N, d, _dtype_code(K),
                                          parent_size, reps_per_parent, _stream(stream),
                                          ctypes.byref(h)))
    return Teams(h, K.dtype)


def kmeans_parents(K: torch.Tensor, parent_size: int, batch_size: int = 4096, max_iter: int = 100,
                   max_no_improvement: int = 10, reassignment_ratio: float = 0.01, init_size: int = 0,
                   seed: int = 0, stream=None):
    """K-means parent labels ``[B, Hkv, N]`` (int32) of prompt keys ``K``;
    returns ``(labels, num_parents, steps)`` with the minibatch steps each
    (b, kv) pair ran."""
    _need(K, "K")
    B, Hkv, N, d = K.shape
    labels = torch.empty((B, Hkv, N), dtype=torch.int32, device=K.device)
    th = _lib.KMeansSettings(batch_size, max_iter, max_no_improvement, float(reassignment_ratio), init_size,
                             seed)
    mp = ctypes.c_int()
    steps = (ctypes.c_int * (B * Hkv))()
    check(_lib.load().santapp_kmeans_parents(_ptr(K), B, Hkv, N, d, _dtype_code(K), parent_size,
                                             ctypes.byref(th), _ptr(labels), ctypes.byref(mp), steps,
                                             _stream(stream)))
    return labels, mp.value, list(steps)


def build_teams_from_labels(K: torch.Tensor, V: torch.Tensor, labels: torch.Tensor, num_labels: int,
                            reps_per_parent: int, stream=None) -> Teams:
    """Team table of the parents ``{i : labels[b, kv, i] == u}``."""
    _need(K, "K")
    _need(V, "V", shape=K.shape, dtype=K.dtype)
    B, Hkv, N, d = K.shape
    _need(labels, "labels", shape=(B, Hkv, N), dtype=torch.int32)
    h = ctypes.c_void_p()
    check(_lib.load().santapp_build_teams_from_labels(_ptr(K), _ptr(V), B, Hkv, N, d, _dtype_code(K),
                                                      _ptr(labels), num_labels, reps_per_parent,
                                                      _stream(stream), ctypes.byref(h)))
    return Teams(h, K.dtype)


def set_route_keys(teams: Teams, kind: str, stream=None) -> None:
    """Route the teams by ``"representative"`` keys (the default after
    :func:`build_teams`) or by ``"centroid"`` keys (team means)."""
    code = {"representative": _lib.ROUTE_REPRESENTATIVE, "centroid": _lib.ROUTE_CENTROID}[kind]
    check(_lib.load().santapp_teams_set_route_keys(teams.handle, code, _stream(stream)))


def routing_kl_workspace(teams: Teams, Hq: int) -> torch.Tensor:
    n = ctypes.c_size_t()
    check(_lib.load().santapp_routing_kl_workspace_bytes(teams.handle, Hq, ctypes.byref(n)))
    return torch.empty(max(n.value, 1), dtype=torch.uint8, device="cuda")


def routing_kl(teams: Teams, q: torch.Tensor, scale: float = 0.0, out: Optional[torch.Tensor] = None,
               workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """KL(p || q) per (sequence, query head) in nats, ``[B, Hq]`` fp64 (eq.
    diagnostic-kl with the table's current routing keys)."""
    _need(q, "q", dtype=torch.float32)
    B, Hq, d = q.shape
    if out is None:
        out = torch.empty((B, Hq), dtype=torch.float64, device="cuda")
    _need(out, "out", shape=(B, Hq), dtype=torch.float64)
    if workspace is None:
        workspace = routing_kl_workspace(teams, Hq)
    check(_lib.load().santapp_routing_kl(teams.handle, _ptr(q), Hq, float(scale), _ptr(out), _ptr(workspace),
                                         workspace.numel(), _stream(stream)))
    return out


def budget_to_K(S: int, P: int, R: int, M: int) -> int:
    k = ctypes.c_int()
    check(_lib.load().santapp_budget_to_K(S, P, R, M, ctypes.byref(k)))
    return k.value


def decode_launch_info(teams: Teams, Hq: int, T: int, K: int) -> tuple:
    """(kernel launches of one step, workgroups of its main launch) for these
    sizes (santapp_decode_launch_info)."""
    k, w = ctypes.c_int(), ctypes.c_int()
    check(_lib.load().santapp_decode_launch_info(teams.handle, Hq, T, K, ctypes.byref(k), ctypes.byref(w)))
    return k.value, w.value


def decode_workspace(teams: Teams, Hq: int, T: int, K: int) -> torch.Tensor:
    n = ctypes.c_size_t()
    check(_lib.load().santapp_decode_workspace_bytes(teams.handle, Hq, T, K, ctypes.byref(n)))
    ws = torch.empty(max(n.value, 1), dtype=torch.uint8, device="cuda")
    check(_lib.load().santapp_workspace_zero(_ptr(ws), n.value, _stream()))
    return ws


def dense_workspace(B: int, Hq: int, Hkv: int, N: int, T: int, d: int) -> torch.Tensor:
    n = ctypes.c_size_t()
    check(_lib.load().santapp_dense_workspace_bytes(B, Hq, Hkv, N, T, d, ctypes.byref(n)))
    ws = torch.empty(max(n.value, 1), dtype=torch.uint8, device="cuda")
    check(_lib.load().santapp_workspace_zero(_ptr(ws), n.value, _stream()))
    return ws


class DebugOut:
    """Device buffers for the optional diagnostics of :func:`decode`."""

    def __init__(self, B: int, Hq: int, Hkv: int, M: int, K: int, arrays: bool = True,
                 events: bool = False):
        dev = "cuda"
        self.phi = self.Y = self.sel = self.logc = self.tau = None
        self.union_teams = self.union_rows = None
        if arrays:
            self.phi = torch.zeros((B, Hq, M), dtype=torch.float64, device=dev)
            self.Y = torch.zeros((B, Hq, M), dtype=torch.float64, device=dev)
            self.sel = torch.full((B, Hq, K), -1, dtype=torch.int32, device=dev)
            self.logc = torch.zeros((B, Hq, K), dtype=torch.float32, device=dev)
            self.tau = torch.zeros((B, Hq), dtype=torch.float64, device=dev)
            self.union_teams = torch.zeros((B, Hkv), dtype=torch.int32, device=dev)
            self.union_rows = torch.zeros((B, Hkv), dtype=torch.int32, device=dev)
        self.events = None
        self.raw_events = None  # caller-created hipEvent_t handles (ctypes.c_void_p)
        if events:
            # torch creates the underlying HIP event at its first record
            self.events = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
            for ev in self.events:
                ev.record()

    def stage_ms(self):
        """(sampling, attention, merge) times of the last call, in ms."""
        e = self.events
        return (e[0].elapsed_time(e[1]), e[1].elapsed_time(e[2]), e[2].elapsed_time(e[3]))

    def struct(self) -> _lib.DecodeDebug:
        def p(t):
            return t.data_ptr() if t is not None else None
        d = _lib.DecodeDebug(p(self.phi), p(self.Y), p(self.sel), p(self.logc), p(self.tau),
                             p(self.union_teams), p(self.union_rows))
        if self.events is not None:
            for i, ev in enumerate(self.events):
                d.events[i] = ev.cuda_event
        if self.raw_events is not None:
            for i, ev in enumerate(self.raw_events):
                d.events[i] = ev.value
        return d


def _suffix(suffix_K, suffix_V, B, Hkv, d, dtype, T=None):
    """Validate a suffix buffer ``[B, Hkv, capacity, d]`` of which the first
    ``T`` rows per (b, kv) are attended (all of them when ``T`` is None);
    returns ``(T, stride)``."""
    if suffix_K is None:
        if T:
            raise SantappError(_lib.EINVAL, "suffix rows requested without a suffix buffer")
        return 0, 0
    cap = suffix_K.shape[2]
    _need(suffix_K, "suffix_K", shape=(B, Hkv, cap, d), dtype=dtype)
    _need(suffix_V, "suffix_V", shape=suffix_K.shape, dtype=dtype)
    T = cap if T is None else int(T)
    if T < 0 or T > cap:
        raise SantappError(_lib.EINVAL, f"T={T} outside the suffix buffer's {cap} rows")
    return T, cap


def decode(teams: Teams, q: torch.Tensor, suffix_K: Optional[torch.Tensor],
           suffix_V: Optional[torch.Tensor], K: int, seed: int = 0, step: int = 0,
           scale: float = 0.0, out: Optional[torch.Tensor] = None,
           workspace: Optional[torch.Tensor] = None, debug: Optional[DebugOut] = None,
           stream=None, T: Optional[int] = None) -> torch.Tensor:
    """One SANTA++ decode step: ``q [B, Hq, d]`` fp32 -> ``out [B, Hq, d]`` fp32.

    ``suffix_K``/``suffix_V`` ``[B, Hkv, capacity, d]`` hold the generated
    rows; the first ``T`` of each (b, kv) are attended (default: all)."""
    B, Hq, d = q.shape
    _need(q, "q", shape=(teams.B, Hq, teams.d), dtype=torch.float32)
    T, stride = _suffix(suffix_K, suffix_V, teams.B, teams.Hkv, teams.d, teams.torch_dtype, T)
    if out is None:
        out = torch.empty((B, Hq, d), dtype=torch.float32, device=q.device)
    _need(out, "out", shape=(B, Hq, d), dtype=torch.float32)
    if workspace is None:
        workspace = decode_workspace(teams, Hq, T, K)
    dbg = ctypes.byref(debug.struct()) if debug is not None else None
    check(_lib.load().santapp_decode(
        teams.handle, _ptr(q), _ptr(suffix_K), _ptr(suffix_V), T, stride, Hq, K,
        ctypes.c_uint64(seed), ctypes.c_uint64(step), float(scale), _ptr(out), _ptr(workspace),
        workspace.numel(), dbg, _stream(stream)))
    return out


def decode_static(teams: Teams, q: torch.Tensor, suffix_K: Optional[torch.Tensor],
                  suffix_V: Optional[torch.Tensor], K: int, out: torch.Tensor, seed: int = 0, step: int = 0,
                  scale: float = 0.0, debug: Optional[DebugOut] = None, stream=None,
                  T: Optional[int] = None) -> torch.Tensor:
    """:func:`decode` over the library's static scratch (santapp_decode_static):
    nothing is allocated, so ``out [B, Hq, d]`` fp32 must be given.  Calls on
    one GPU share the scratch and must not overlap in time."""
    B, Hq, d = q.shape
    _need(q, "q", shape=(teams.B, Hq, teams.d), dtype=torch.float32)
    T, stride = _suffix(suffix_K, suffix_V, teams.B, teams.Hkv, teams.d, teams.torch_dtype, T)
    _need(out, "out", shape=(B, Hq, d), dtype=torch.float32)
    dbg = ctypes.byref(debug.struct()) if debug is not None else None
    check(_lib.load().santapp_decode_static(
        teams.handle, _ptr(q), _ptr(suffix_K), _ptr(suffix_V), T, stride, Hq, K,
        ctypes.c_uint64(seed), ctypes.c_uint64(step), float(scale), _ptr(out), dbg, _stream(stream)))
    return out


def dense_decode(q: torch.Tensor, K: torch.Tensor, V: torch.Tensor,
                 suffix_K: Optional[torch.Tensor], suffix_V: Optional[torch.Tensor],
                 scale: float = 0.0, out: Optional[torch.Tensor] = None,
                 workspace: Optional[torch.Tensor] = None, stream=None,
                 T: Optional[int] = None, debug: Optional[DebugOut] = None) -> torch.Tensor:
    """Dense attention over K, V ``[B, Hkv, N, d]`` plus the first ``T`` suffix
    rows of ``[B, Hkv, capacity, d]`` (default: all).  ``debug``: only its
    stage events are used."""
    B, Hq, d = q.shape
    _need(q, "q", dtype=torch.float32)
    _need(K, "K")
    _need(V, "V", shape=K.shape, dtype=K.dtype)
    _, Hkv, N, _ = K.shape
    T, stride = _suffix(suffix_K, suffix_V, B, Hkv, d, K.dtype, T)
    if out is None:
        out = torch.empty((B, Hq, d), dtype=torch.float32, device=q.device)
    if workspace is None:
        workspace = dense_workspace(B, Hq, Hkv, N, T, d)
    dbg = ctypes.byref(debug.struct()) if debug is not None else None
    check(_lib.load().santapp_dense_decode(
        _ptr(q), _ptr(K), _ptr(V), B, Hkv, N, d, _dtype_code(K), _ptr(suffix_K), _ptr(suffix_V),
        T, stride, Hq, float(scale), _ptr(out), _ptr(workspace), workspace.numel(), dbg, _stream(stream)))
    return out
