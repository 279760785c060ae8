"""ctypes binding of libecmoe.so (see include/ec_moe.h for the contract).

Argument marshalling only: shapes and dtypes are read off torch tensors, the
workspace is a torch allocation, and every call is enqueued on torch's
current HIP stream.  The library is loaded on first use and a missing or
stale build raises instead of falling back to anything.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libecmoe.so")

EC_F32, EC_BF16 = 0, 1
SCHEDULERS = {"linear": 0, "linear_rev": 1, "cosine": 2, "cosine_rev": 3, "gaussian": 4,
              "gaussian_rev": 5}
EXPORTS = ("ec_status_string", "ec_last_error", "ec_total_capacity", "ec_workspace_size",
           "ec_saved_size", "ec_saved_layout_of", "ec_capacity", "ec_route", "ec_route_noalloc", "ec_token_coverage", "ec_moe_forward",
           "ec_moe_backward", "ec_tc_capacity", "ec_tc_workspace_size", "ec_tc_route",
           "ec_tc_forward", "ec_set_stage_events")


class ECError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(msg)
        self.status = status


class _Problem(ctypes.Structure):
    _fields_ = [("n_tokens", ctypes.c_int64), ("d_model", ctypes.c_int32),
                ("n_experts", ctypes.c_int32), ("d_ff", ctypes.c_int32),
                ("n_groups", ctypes.c_int32), ("group_offsets", ctypes.POINTER(ctypes.c_int32)),
                ("capacity", ctypes.POINTER(ctypes.c_int32)), ("inv_temperature", ctypes.c_float),
                ("dtype", ctypes.c_int), ("d_shared", ctypes.c_int32)]


class _SavedLayout(ctypes.Structure):
    _fields_ = [(n, ctypes.c_size_t) for n in ("S", "sel_token", "sel_gate", "slot", "Xe", "H1",
                                               "H3", "A", "O", "Hs1", "Hs3", "As", "total")]


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2604_01622_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        vp, sz, i32p = ctypes.c_void_p, ctypes.c_size_t, ctypes.POINTER(ctypes.c_int32)
        pp = ctypes.POINTER(_Problem)
        L.ec_status_string.restype = ctypes.c_char_p
        L.ec_status_string.argtypes = [ctypes.c_int]
        L.ec_last_error.restype = ctypes.c_char_p
        L.ec_last_error.argtypes = []
        L.ec_total_capacity.restype = ctypes.c_int64
        L.ec_total_capacity.argtypes = [pp]
        L.ec_workspace_size.restype = sz
        L.ec_workspace_size.argtypes = [pp, ctypes.c_int]
        L.ec_saved_size.restype = sz
        L.ec_saved_size.argtypes = [pp]
        L.ec_saved_layout_of.restype = ctypes.c_int
        L.ec_saved_layout_of.argtypes = [pp, ctypes.POINTER(_SavedLayout)]
        L.ec_capacity.restype = ctypes.c_int
        L.ec_capacity.argtypes = [ctypes.c_int32, i32p, ctypes.c_int32, ctypes.c_double,
                                  ctypes.POINTER(ctypes.c_double), ctypes.c_double,
                                  ctypes.c_double, ctypes.c_int, i32p]
        L.ec_route.restype = ctypes.c_int
        L.ec_route.argtypes = [pp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.ec_route_noalloc.restype = ctypes.c_int
        L.ec_route_noalloc.argtypes = [pp, vp, vp, vp, vp, vp, vp, vp]
        L.ec_token_coverage.restype = ctypes.c_int
        L.ec_token_coverage.argtypes = [pp, vp, vp, vp, vp]
        L.ec_moe_forward.restype = ctypes.c_int
        L.ec_moe_forward.argtypes = [pp] + [vp] * 9 + [vp, sz, vp, sz, vp]
        L.ec_moe_backward.restype = ctypes.c_int
        L.ec_moe_backward.argtypes = [pp] + [vp] * 9 + [vp, sz] + [vp] * 8 + [vp, sz, vp]
        L.ec_tc_capacity.restype = ctypes.c_int
        L.ec_tc_capacity.argtypes = [ctypes.c_int32, i32p, ctypes.c_int32, ctypes.c_int32,
                                     ctypes.c_double, i32p]
        L.ec_tc_workspace_size.restype = sz
        L.ec_tc_workspace_size.argtypes = [pp, ctypes.c_int32, ctypes.c_int]
        L.ec_tc_route.restype = ctypes.c_int
        L.ec_tc_route.argtypes = [pp, ctypes.c_int32] + [vp] * 8 + [sz, vp]
        L.ec_tc_forward.restype = ctypes.c_int
        L.ec_tc_forward.argtypes = [pp, ctypes.c_int32] + [vp] * 11 + [sz, vp]
        L.ec_set_stage_events.restype = ctypes.c_int
        L.ec_set_stage_events.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_int]
        _lib = L
    return _lib


def _check(status: int):
    if status != 0:
        L = lib()
        raise ECError(status, f"{L.ec_status_string(status).decode()}: "
                              f"{L.ec_last_error().decode()}")


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dtype_code(dt: torch.dtype) -> int:
    if dt == torch.bfloat16:
        return EC_BF16
    if dt == torch.float32:
        return EC_F32
    raise ECError(4, f"unsupported storage dtype {dt}")


class Problem:
    """Host-side problem description (group offsets and capacities stay on the host)."""

    def __init__(self, n_tokens: int, d_model: int, n_experts: int, d_ff: int,
                 group_offsets: Sequence[int], capacity: Sequence[int], inv_temperature: float,
                 dtype: torch.dtype, d_shared: int = 0):
        self.off = np.ascontiguousarray(np.asarray(group_offsets, dtype=np.int32))
        self.cap = np.ascontiguousarray(np.asarray(capacity, dtype=np.int32))
        self.dtype = dtype
        self.c = _Problem(int(n_tokens), int(d_model), int(n_experts), int(d_ff),
                          int(len(self.cap)),
                          self.off.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                          self.cap.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                          float(inv_temperature), _dtype_code(dtype), int(d_shared))

    @property
    def ref(self):
        return ctypes.byref(self.c)

    @property
    def K(self) -> int:
        k = lib().ec_total_capacity(self.ref)
        if k < 0:
            raise ECError(2, lib().ec_last_error().decode())
        return int(k)

    def workspace_size(self, mode: int) -> int:
        n = lib().ec_workspace_size(self.ref, mode)
        if n == 0:
            msg = lib().ec_last_error().decode()
            if msg:
                raise ECError(1, msg)
        return int(n)

    def saved_size(self) -> int:
        n = lib().ec_saved_size(self.ref)
        if n == 0:
            raise ECError(2, lib().ec_last_error().decode())
        return int(n)

    def saved_layout(self) -> dict:
        lay = _SavedLayout()
        _check(lib().ec_saved_layout_of(self.ref, ctypes.byref(lay)))
        return {n: getattr(lay, n) for n, _ in _SavedLayout._fields_}

    @staticmethod
    def of(X: torch.Tensor, Wg: torch.Tensor, d_ff: int, group_offsets, capacity,
           inv_temperature: float = 1.0, shared=None) -> "Problem":
        return Problem(X.shape[0], X.shape[1], Wg.shape[0], d_ff, group_offsets, capacity,
                       inv_temperature, X.dtype, 0 if shared is None else shared[0].shape[0])


def _empty(nbytes: int, device) -> torch.Tensor:
    return torch.empty(max(int(nbytes), 16), dtype=torch.uint8, device=device)


def capacity(group_lengths: Sequence[int], n_experts: int, c: Optional[float] = None,
             t: Optional[Sequence[float]] = None, c_min: float = 0.0, c_max: float = 0.0,
             scheduler: str = "linear_rev") -> np.ndarray:
    """Tokens per expert in each group (library's ec_capacity)."""
    L = np.ascontiguousarray(np.asarray(group_lengths, dtype=np.int32))
    out = np.zeros(len(L), dtype=np.int32)
    tp = None
    if t is not None:
        tt = np.ascontiguousarray(np.asarray(t, dtype=np.float64))
        tp = tt.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
    _check(lib().ec_capacity(len(L), L.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)),
                             int(n_experts), float(c if c is not None else 0.0), tp,
                             float(c_min), float(c_max), SCHEDULERS[scheduler],
                             out.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))))
    return out


def route(X: torch.Tensor, Wg: torch.Tensor, group_offsets, capacity, inv_temperature=1.0,
          d_ff: int = 64):
    """Router + column top-k.  Returns S [N,E] fp32, sel_token [E,K] int32,
    sel_gate [E,K] fp32 and slot [E,N] int32."""
    P = Problem.of(X, Wg, d_ff, group_offsets, capacity, inv_temperature)
    N, E, K = X.shape[0], Wg.shape[0], P.K
    dev = X.device
    S = torch.empty((N, E), dtype=torch.float32, device=dev)
    sel = torch.empty((E, K), dtype=torch.int32, device=dev)
    gate = torch.empty((E, K), dtype=torch.float32, device=dev)
    slot = torch.empty((E, N), dtype=torch.int32, device=dev)
    ws = _empty(P.workspace_size(0), dev)
    _check(lib().ec_route(P.ref, _ptr(X), _ptr(Wg), _ptr(S), _ptr(sel) if K else None,
                          _ptr(gate) if K else None, _ptr(slot), _ptr(ws), ws.numel(),
                          _stream()))
    return S, sel, gate, slot


def route_noalloc(X: torch.Tensor, Wg: torch.Tensor, group_offsets, capacity,
                  inv_temperature=1.0, d_ff: int = 64, with_slot: bool = True):
    """Router + column top-k with the library's static scratch instead of a
    workspace (ec_route_noalloc).  Returns S, sel_token, sel_gate and slot (None
    when with_slot is False: the slot map then lives in the scratch)."""
    P = Problem.of(X, Wg, d_ff, group_offsets, capacity, inv_temperature)
    N, E, K = X.shape[0], Wg.shape[0], P.K
    dev = X.device
    S = torch.empty((N, E), dtype=torch.float32, device=dev)
    sel = torch.empty((E, K), dtype=torch.int32, device=dev)
    gate = torch.empty((E, K), dtype=torch.float32, device=dev)
    slot = torch.empty((E, N), dtype=torch.int32, device=dev) if with_slot else None
    _check(lib().ec_route_noalloc(P.ref, _ptr(X), _ptr(Wg), _ptr(S), _ptr(sel) if K else None,
                                  _ptr(gate) if K else None, _ptr(slot), _stream()))
    return S, sel, gate, slot


def token_coverage(slot: torch.Tensor, group_offsets, capacity, d_model: int = 64,
                   d_ff: int = 64):
    """Token drop statistic from a slot map [E,N] int32.  Returns experts_per_token [N]
    int32 and dropped [G] int32 (tokens of each group that no expert chose)."""
    E, N = slot.shape
    off = np.asarray(group_offsets, dtype=np.int64)
    P = Problem(N, d_model, E, d_ff, off, capacity, 1.0, torch.bfloat16)
    cnt = torch.empty((N,), dtype=torch.int32, device=slot.device)
    dropped = torch.empty((len(off) - 1,), dtype=torch.int32, device=slot.device)
    _check(lib().ec_token_coverage(P.ref, _ptr(slot) if N else None, _ptr(cnt) if N else None,
                                   _ptr(dropped), _stream()))
    return cnt, dropped


def tc_capacity(group_lengths: Sequence[int], n_experts: int, top_k: int,
                cf: float) -> np.ndarray:
    """Token-choice capacity per (group, expert): min(L_g, ceil(cf k L_g / E)); cf <= 0: no cap."""
    L = np.ascontiguousarray(np.asarray(group_lengths, dtype=np.int32))
    out = np.empty(len(L), dtype=np.int32)
    i32p = ctypes.POINTER(ctypes.c_int32)
    _check(lib().ec_tc_capacity(len(L), L.ctypes.data_as(i32p), int(n_experts), int(top_k),
                                float(cf), out.ctypes.data_as(i32p)))
    return out


def _tc_rmax(P: "Problem", top_k: int) -> int:
    N, E = P.c.n_tokens, P.c.n_experts
    return int(min(top_k * N, E * min(int(P.cap.sum()), N)))


def tc_route(X, Wg, group_offsets, capacity, top_k: int, inv_temperature=1.0, d_ff: int = 64):
    """Token-choice routing.  Returns S [N,E], G [N,E] (gates of kept pairs), slot [E,N]
    (packed row or -1), expert_rows [E+1] and sel_token (token of each packed row)."""
    P = Problem.of(X, Wg, d_ff, group_offsets, capacity, inv_temperature)
    N, E = X.shape[0], Wg.shape[0]
    dev = X.device
    S = torch.empty((N, E), dtype=torch.float32, device=dev)
    G = torch.empty((N, E), dtype=torch.float32, device=dev)
    slot = torch.empty((E, N), dtype=torch.int32, device=dev)
    rows = torch.empty((E + 1,), dtype=torch.int32, device=dev)
    sel = torch.empty((max(_tc_rmax(P, top_k), 1),), dtype=torch.int32, device=dev)
    n = lib().ec_tc_workspace_size(P.ref, int(top_k), 0)
    if n == 0:
        _check(2)
    ws = _empty(n, dev)
    _check(lib().ec_tc_route(P.ref, int(top_k), _ptr(X), _ptr(Wg), _ptr(S), _ptr(G), _ptr(slot),
                             _ptr(rows), _ptr(sel), _ptr(ws), ws.numel(), _stream()))
    return S, G, slot, rows, sel


def tc_forward(X, Wg, W1, W3, W2, group_offsets, capacity, top_k: int, inv_temperature=1.0,
               shared=None):
    """Token-choice layer forward.  Returns Y [N,d] and expert_rows [E+1]."""
    P = Problem.of(X, Wg, W1.shape[1], group_offsets, capacity, inv_temperature, shared)
    dev = X.device
    Y = torch.empty_like(X)
    rows = torch.empty((Wg.shape[0] + 1,), dtype=torch.int32, device=dev)
    n = lib().ec_tc_workspace_size(P.ref, int(top_k), 1)
    if n == 0:
        _check(2)
    ws = _empty(n, dev)
    _check(lib().ec_tc_forward(P.ref, int(top_k), _ptr(X), _ptr(Wg), _ptr(W1), _ptr(W3), _ptr(W2),
                               *_shared_ptrs(shared), _ptr(Y), _ptr(rows), _ptr(ws), ws.numel(),
                               _stream()))
    return Y, rows


def _shared_ptrs(shared):
    return [None, None, None] if shared is None else [_ptr(w) for w in shared]


def forward(X, Wg, W1, W3, W2, group_offsets, capacity, inv_temperature=1.0, save=False,
            shared=None):
    """Layer forward.  shared: (Ws1 [hs,d], Ws3 [hs,d], Ws2 [d,hs]) of the shared experts or
    None.  Returns Y [N,d] (and the saved-activation buffer if save)."""
    P = Problem.of(X, Wg, W1.shape[1], group_offsets, capacity, inv_temperature, shared)
    dev = X.device
    Y = torch.empty_like(X)
    saved = _empty(P.saved_size(), dev) if save else None
    ws = _empty(P.workspace_size(3 if save else 1), dev)
    _check(lib().ec_moe_forward(P.ref, _ptr(X), _ptr(Wg), _ptr(W1), _ptr(W3), _ptr(W2),
                                *_shared_ptrs(shared), _ptr(Y), _ptr(saved),
                                0 if saved is None else saved.numel(), _ptr(ws), ws.numel(),
                                _stream()))
    return (Y, saved) if save else Y


def backward(X, Wg, W1, W3, W2, dY, saved, group_offsets, capacity, inv_temperature=1.0,
             shared=None):
    """Layer backward.  Returns dX, dWg (fp32), dW1, dW3, dW2 (and dWs1, dWs3, dWs2 with
    shared experts)."""
    P = Problem.of(X, Wg, W1.shape[1], group_offsets, capacity, inv_temperature, shared)
    dev = X.device
    dX = torch.empty_like(X)
    dWg = torch.empty(Wg.shape, dtype=torch.float32, device=dev)
    dW1, dW3, dW2 = torch.empty_like(W1), torch.empty_like(W3), torch.empty_like(W2)
    dsh = None if shared is None else [torch.empty_like(w) for w in shared]
    ws = _empty(P.workspace_size(2), dev)
    _check(lib().ec_moe_backward(P.ref, _ptr(X), _ptr(Wg), _ptr(W1), _ptr(W3), _ptr(W2),
                                 *_shared_ptrs(shared), _ptr(dY), _ptr(saved), saved.numel(),
                                 _ptr(dX), _ptr(dWg), _ptr(dW1), _ptr(dW3), _ptr(dW2),
                                 *_shared_ptrs(dsh), _ptr(ws), ws.numel(), _stream()))
    if shared is None:
        return dX, dWg, dW1, dW3, dW2
    return (dX, dWg, dW1, dW3, dW2) + tuple(dsh)


def saved_views(saved: torch.Tensor, P: Problem) -> dict:
    """Typed views into a saved-activation buffer (S, sel_token, sel_gate, slot, Xe (fp32
    only), H1, H3, A (gate-scaled), O (gate-weighted) and the shared experts' activations)."""
    lay = P.saved_layout()
    N, d, E, h, K = P.c.n_tokens, P.c.d_model, P.c.n_experts, P.c.d_ff, P.K
    dt = P.dtype
    es = 4 if dt == torch.float32 else 2

    def view(off, shape, dtype, esize):
        n = int(np.prod(shape))
        return saved[off:off + n * esize].view(dtype).view(*shape)

    out = {"S": view(lay["S"], (N, E), torch.float32, 4),
            "sel_token": view(lay["sel_token"], (E, K), torch.int32, 4),
            "sel_gate": view(lay["sel_gate"], (E, K), torch.float32, 4),
            "slot": view(lay["slot"], (E, N), torch.int32, 4),
            "H1": view(lay["H1"], (E, K, h), dt, es),
            "H3": view(lay["H3"], (E, K, h), dt, es), "A": view(lay["A"], (E, K, h), dt, es),
            "O": view(lay["O"], (E, K, d), dt, es),
            "Hs1": view(lay["Hs1"], (N, P.c.d_shared), dt, es),
            "Hs3": view(lay["Hs3"], (N, P.c.d_shared), dt, es),
            "As": view(lay["As"], (N, P.c.d_shared), dt, es)}
    if dt == torch.float32:    # fp32 keeps the gathered rows; bf16 reads them from X
        out["Xe"] = view(lay["Xe"], (E, K, d), dt, es)
    return out


class Layer:
    """Pre-planned layer: workspace, saved buffer and outputs allocated once, so
    that repeated calls only enqueue kernels (used by the benchmark)."""

    def __init__(self, X, Wg, W1, W3, W2, group_offsets, capacity, inv_temperature=1.0,
                 training=False, shared=None):
        self.X, self.Wg, self.W1, self.W3, self.W2 = X, Wg, W1, W3, W2
        self.shared = shared
        self.P = Problem.of(X, Wg, W1.shape[1], group_offsets, capacity, inv_temperature, shared)
        dev = X.device
        self.Y = torch.empty_like(X)
        self.saved = _empty(self.P.saved_size(), dev) if training else None
        self.ws_f = _empty(self.P.workspace_size(3 if training else 1), dev)
        if training:
            self.ws_b = _empty(self.P.workspace_size(2), dev)
            self.dX = torch.empty_like(X)
            self.dWg = torch.empty(Wg.shape, dtype=torch.float32, device=dev)
            self.dW1, self.dW3 = torch.empty_like(W1), torch.empty_like(W3)
            self.dW2 = torch.empty_like(W2)
            self.dshared = None if shared is None else [torch.empty_like(w) for w in shared]
        self._fwd_args = None

    def forward(self):
        _check(lib().ec_moe_forward(self.P.ref, _ptr(self.X), _ptr(self.Wg), _ptr(self.W1),
                                    _ptr(self.W3), _ptr(self.W2), *_shared_ptrs(self.shared),
                                    _ptr(self.Y), _ptr(self.saved),
                                    0 if self.saved is None else self.saved.numel(),
                                    _ptr(self.ws_f), self.ws_f.numel(), _stream()))
        return self.Y

    def backward(self, dY):
        _check(lib().ec_moe_backward(self.P.ref, _ptr(self.X), _ptr(self.Wg), _ptr(self.W1),
                                     _ptr(self.W3), _ptr(self.W2), *_shared_ptrs(self.shared),
                                     _ptr(dY), _ptr(self.saved),
                                     self.saved.numel(), _ptr(self.dX), _ptr(self.dWg),
                                     _ptr(self.dW1), _ptr(self.dW3), _ptr(self.dW2),
                                     *_shared_ptrs(self.dshared),
                                     _ptr(self.ws_b), self.ws_b.numel(), _stream()))
        return self.dX, self.dWg, self.dW1, self.dW3, self.dW2


class TcLayer:
    """Pre-planned token-choice forward (the comparison policy): workspace and outputs
    allocated once."""

    def __init__(self, X, Wg, W1, W3, W2, group_offsets, capacity, top_k: int,
                 inv_temperature=1.0, shared=None):
        self.X, self.Wg, self.W1, self.W3, self.W2 = X, Wg, W1, W3, W2
        self.shared = shared
        self.top_k = int(top_k)
        self.P = Problem.of(X, Wg, W1.shape[1], group_offsets, capacity, inv_temperature, shared)
        dev = X.device
        self.Y = torch.empty_like(X)
        self.rows = torch.empty((Wg.shape[0] + 1,), dtype=torch.int32, device=dev)
        n = lib().ec_tc_workspace_size(self.P.ref, self.top_k, 1)
        if n == 0:
            _check(2)
        self.ws = _empty(n, dev)

    def forward(self):
        _check(lib().ec_tc_forward(self.P.ref, self.top_k, _ptr(self.X), _ptr(self.Wg),
                                   _ptr(self.W1), _ptr(self.W3), _ptr(self.W2),
                                   *_shared_ptrs(self.shared), _ptr(self.Y), _ptr(self.rows),
                                   _ptr(self.ws), self.ws.numel(), _stream()))
        return self.Y


FORWARD_STAGES = ("router", "topk", "gather", "gemm_w13_swiglu", "gemm_w2", "shared_w13_swiglu",
                  "shared_w2", "combine")
BACKWARD_STAGES = ("bwd_gather", "gemm_dA_swiglu_bwd", "gemm_dW2", "gemm_dXe", "gemm_dW13",
                   "router_dz", "router_dx", "shared_dA_swiglu_bwd", "shared_dW2", "shared_dX",
                   "shared_dW13", "bwd_combine", "router_dwg")


class StageEvents:
    """torch.cuda.Event objects that the library records between its stages."""

    def __init__(self, n_stages: int):
        self.events = [torch.cuda.Event(enable_timing=True) for _ in range(n_stages + 1)]
        for e in self.events:   # torch creates the underlying HIP event on first record
            e.record()
        self._arr = (ctypes.c_void_p * len(self.events))()

    def arm(self):
        for i, e in enumerate(self.events):
            self._arr[i] = e.cuda_event
        _check(lib().ec_set_stage_events(self._arr, len(self.events)))

    @staticmethod
    def disarm():
        _check(lib().ec_set_stage_events(None, 0))

    def durations_ms(self):
        return [a.elapsed_time(b) for a, b in zip(self.events[:-1], self.events[1:])]
