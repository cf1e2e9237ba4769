"""ctypes binding of ``libmaskmoe.so``: argument marshalling only.

Every function takes torch tensors on the current HIP device, checks their
dtype/shape/contiguity, allocates the outputs with torch (device memory is the
only thing torch provides here) and calls the C entry point of the same name on
torch's current stream. All arithmetic runs in the library's kernels; there is
no fallback of any kind: a missing library raises.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libmaskmoe.so")

OK, E_INVAL, E_WORKSPACE, E_HIP, E_UNSUPPORTED = 0, 1, 2, 3, 4
ROUTE_PLAIN, ROUTE_HARD_MASK, ROUTE_SOFT_PRIOR = 0, 1, 2
GATE_P, GATE_RENORM = 0, 1
BF16, F32 = 0, 1
CACHE_LRU, CACHE_LFU, CACHE_FIFO = 0, 1, 2

EXPORTS = ("maskmoe_route", "maskmoe_layer_workspace_bytes", "maskmoe_layer_forward",
           "maskmoe_layer_forward_profiled", "maskmoe_cache_fetches", "maskmoe_status_string")
NUM_STAGES = 5
STAGES = ("route", "permute", "gate_up", "down", "combine")


class LayerDesc(ctypes.Structure):
    """``maskmoe_layer_desc``."""

    _fields_ = [(n, ctypes.c_int32) for n in
                ("T", "d", "E", "K", "F", "n_shared", "dtype", "route_mode", "gate_mode")]


class MaskMoEError(RuntimeError):
    def __init__(self, fn: str, status: int, text: str):
        super().__init__(f"{fn} failed with status {status} ({text})")
        self.status = status


_lib = None
_vp, _i32, _sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load the library (once). Loud failure when it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with __graft_entry__.build() "
                           "(hipcc --offload-arch=gfx950); there is no fallback path")
    # torch first: its HIP runtime then satisfies the library's libamdhip64 dependency,
    # so the process holds a single HIP runtime.
    import torch  # noqa: F401
    lib = ctypes.CDLL(path)
    lib.maskmoe_route.argtypes = [ctypes.POINTER(LayerDesc), _i32, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp]
    lib.maskmoe_route.restype = ctypes.c_int
    lib.maskmoe_layer_workspace_bytes.argtypes = [ctypes.POINTER(LayerDesc)]
    lib.maskmoe_layer_workspace_bytes.restype = _sz
    lib.maskmoe_layer_forward.argtypes = [ctypes.POINTER(LayerDesc), _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                          _vp, _vp, _vp, _vp, _sz, _vp]
    lib.maskmoe_layer_forward.restype = ctypes.c_int
    lib.maskmoe_layer_forward_profiled.argtypes = [ctypes.POINTER(LayerDesc), _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                                   _vp, _vp, _vp, _vp, _vp, _sz, _vp, _vp]
    lib.maskmoe_layer_forward_profiled.restype = ctypes.c_int
    lib.maskmoe_cache_fetches.argtypes = [_vp, _i32, _i32, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp,
                                          _vp, _vp, _vp, _vp]
    lib.maskmoe_cache_fetches.restype = ctypes.c_int
    lib.maskmoe_status_string.argtypes = [ctypes.c_int]
    lib.maskmoe_status_string.restype = ctypes.c_char_p
    _lib = lib
    return lib


def _check(fn: str, status: int) -> None:
    if status != OK:
        raise MaskMoEError(fn, status, load().maskmoe_status_string(status).decode())


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream():
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return BF16
    if t.dtype == torch.float32:
        return F32
    raise TypeError(f"unsupported dtype {t.dtype}: use bfloat16 or float32")


def _dev(t, name: str):
    if t is None:
        return
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _host_u8(a, n: int):
    if a is None:
        return None, None
    arr = np.ascontiguousarray(np.asarray(a.cpu() if hasattr(a, "cpu") else a).reshape(-1), dtype=np.uint8)
    if arr.size != n:
        raise ValueError(f"mask has {arr.size} entries, expected {n}")
    return arr, arr.ctypes.data_as(ctypes.c_void_p)


def _host_f32(a, n: int):
    if a is None:
        return None, None
    arr = np.ascontiguousarray(np.asarray(a.cpu() if hasattr(a, "cpu") else a).reshape(-1), dtype=np.float32)
    if arr.size != n:
        raise ValueError(f"prior has {arr.size} entries, expected {n}")
    return arr, arr.ctypes.data_as(ctypes.c_void_p)


def make_desc(T, d, E, K, F=1, n_shared=0, dtype=BF16, route_mode=ROUTE_PLAIN, gate_mode=GATE_RENORM) -> LayerDesc:
    return LayerDesc(T, d, E, K, F, n_shared, dtype, route_mode, gate_mode)


def maskmoe_route(x, w_router, K: int, route_mode: int, gate_mode: int, mask=None, prior=None,
                  with_margin: bool = True):
    """Route tokens x [T,d] through L routers w_router [L,E,d] (or [E,d] for L=1).

    mask / prior: host arrays [L,E] (or [E]). Returns ``(idx [L,T,K] int32,
    gate [L,T,K] float32, margin [L,T] float32 or None)``; L is squeezed when
    ``w_router`` is 2-D.
    """
    import torch
    lib = load()
    _dev(x, "x")
    _dev(w_router, "w_router")
    squeeze = w_router.dim() == 2
    w3 = w_router.unsqueeze(0) if squeeze else w_router
    L, E, d = w3.shape
    T = x.shape[0]
    if x.shape[1] != d or x.dtype != w3.dtype:
        raise ValueError("x and w_router disagree in hidden size or dtype")
    desc = make_desc(T, d, E, K, dtype=_dtype_code(x), route_mode=route_mode, gate_mode=gate_mode)
    m_arr, m_p = _host_u8(mask, L * E) if route_mode == ROUTE_HARD_MASK else (None, None)
    p_arr, p_p = _host_f32(prior, L * E) if route_mode == ROUTE_SOFT_PRIOR else (None, None)
    idx = torch.empty((L, T, K), dtype=torch.int32, device=x.device)
    gate = torch.empty((L, T, K), dtype=torch.float32, device=x.device)
    margin = torch.empty((L, T), dtype=torch.float32, device=x.device) if with_margin else None
    _check("maskmoe_route", lib.maskmoe_route(ctypes.byref(desc), L, _ptr(x), _ptr(w3), m_p, p_p, _ptr(idx),
                                              _ptr(gate), _ptr(margin), _stream()))
    del m_arr, p_arr
    if squeeze:
        return idx[0], gate[0], (margin[0] if margin is not None else None)
    return idx, gate, margin


def maskmoe_layer_workspace_bytes(desc: LayerDesc) -> int:
    return int(load().maskmoe_layer_workspace_bytes(ctypes.byref(desc)))


def maskmoe_layer_forward(x, w_router, w_gate_up, w_down, K: int, route_mode: int, gate_mode: int,
                          mask=None, prior=None, ws_gate_up=None, ws_down=None, workspace=None, y=None,
                          topk_idx=None, topk_gate=None, events=None):
    """One masked MoE layer. Shapes: x [T,d], w_router [E,d], w_gate_up [E,2F,d],
    w_down [E,d,F], ws_gate_up [S,2F,d], ws_down [S,d,F]; mask/prior host [E].

    Returns y [T,d] (dtype of x). ``workspace`` (uint8 device tensor) is
    allocated when not given; ``topk_idx``/``topk_gate`` [T,K] receive the
    routing decision when given. ``events``: NUM_STAGES + 1 entries, each None or an
    already-recorded ``torch.cuda.Event(enable_timing=True)``; when given, the
    profiled entry point re-records the non-None ones around the stages.
    """
    import torch
    lib = load()
    for t, n in ((x, "x"), (w_router, "w_router"), (w_gate_up, "w_gate_up"), (w_down, "w_down"),
                 (ws_gate_up, "ws_gate_up"), (ws_down, "ws_down"), (y, "y"), (workspace, "workspace"),
                 (topk_idx, "topk_idx"), (topk_gate, "topk_gate")):
        _dev(t, n)
    T, d = x.shape
    E, F2, d2 = w_gate_up.shape
    F = F2 // 2
    if d2 != d or tuple(w_down.shape) != (E, d, F) or tuple(w_router.shape) != (E, d):
        raise ValueError("inconsistent layer shapes")
    ns = 0 if ws_gate_up is None else ws_gate_up.shape[0]
    if ns and (tuple(ws_gate_up.shape) != (ns, 2 * F, d) or tuple(ws_down.shape) != (ns, d, F)):
        raise ValueError("inconsistent shared-expert shapes")
    for t in (w_router, w_gate_up, w_down, ws_gate_up, ws_down):
        if t is not None and t.dtype != x.dtype:
            raise ValueError("all weights must have the dtype of x")
    desc = make_desc(T, d, E, K, F, ns, _dtype_code(x), route_mode, gate_mode)
    need = maskmoe_layer_workspace_bytes(desc)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
    if y is None:
        y = torch.empty((T, d), dtype=x.dtype, device=x.device)
    m_arr, m_p = _host_u8(mask, E) if route_mode == ROUTE_HARD_MASK else (None, None)
    p_arr, p_p = _host_f32(prior, E) if route_mode == ROUTE_SOFT_PRIOR else (None, None)
    args = (ctypes.byref(desc), _ptr(x), _ptr(w_router), m_p, p_p, _ptr(w_gate_up), _ptr(w_down),
            _ptr(ws_gate_up), _ptr(ws_down), _ptr(y), _ptr(topk_idx), _ptr(topk_gate), _ptr(workspace),
            workspace.numel())
    if events is None:
        _check("maskmoe_layer_forward", lib.maskmoe_layer_forward(*args, _stream()))
    else:
        if len(events) != NUM_STAGES + 1:
            raise ValueError(f"need {NUM_STAGES + 1} events")
        handles = (ctypes.c_void_p * len(events))(*[None if ev is None else ev.cuda_event for ev in events])
        _check("maskmoe_layer_forward_profiled", lib.maskmoe_layer_forward_profiled(*args, handles, _stream()))
    del m_arr, p_arr
    return y


def maskmoe_cache_fetches(trace, E: int, B: int, state=None, with_f_per_step: bool = False,
                          dev_error=None, policy: int = CACHE_LRU, counts=None):
    """Replay traces [L,S,N,K] (int32 device) through per-(layer, stream) caches under
    ``policy`` (CACHE_LRU, CACHE_LFU or CACHE_FIFO); ``counts`` [L,S,E] int32 device holds
    LFU access counts (in/out) or is None.

    ``state`` [L,S,B] int32 device (in/out) or None; ``dev_error`` an int32
    device tensor that the kernel sets to 1 when it skips an entry (never
    cleared), or None. Returns a dict with ``fetches``/``hits`` [L,S] int64,
    ``f_per_step`` [L,S,N] uint8 (or None) and ``dev_error``.
    """
    import torch
    lib = load()
    _dev(trace, "trace")
    _dev(state, "state")
    if trace.dtype != torch.int32 or trace.dim() != 4:
        raise ValueError("trace must be int32 [L,S,N,K]")
    L, S, N, K = trace.shape
    dev = trace.device
    fetches = torch.empty((L, S), dtype=torch.int64, device=dev)
    hits = torch.empty((L, S), dtype=torch.int64, device=dev)
    fps = torch.empty((L, S, N), dtype=torch.uint8, device=dev) if with_f_per_step else None
    if state is not None and (state.dtype != torch.int32 or tuple(state.shape) != (L, S, B)):
        raise ValueError("state must be int32 [L,S,B]")
    _dev(counts, "counts")
    if counts is not None and (counts.dtype != torch.int32 or tuple(counts.shape) != (L, S, E)):
        raise ValueError("counts must be int32 [L,S,E]")
    _check("maskmoe_cache_fetches", lib.maskmoe_cache_fetches(
        _ptr(trace), L, S, N, K, E, B, policy, _ptr(state), _ptr(counts), _ptr(fetches), _ptr(hits), _ptr(fps),
        _ptr(dev_error), _stream()))
    return {"fetches": fetches, "hits": hits, "f_per_step": fps, "dev_error": dev_error}
