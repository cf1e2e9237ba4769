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
LAYOUT_ROWS, LAYOUT_PACKED = 0, 1

EXPORTS = ("maskmoe_route", "maskmoe_route_workspace_bytes", "maskmoe_layer_workspace_bytes",
           "maskmoe_layer_forward", "maskmoe_layer_forward_profiled", "maskmoe_cache_fetches", "maskmoe_status_string",
           "maskmoe_sample_mask", "maskmoe_layer_forward_train", "maskmoe_stage1_backward_workspace_bytes",
           "maskmoe_stage1_backward", "maskmoe_layer_train_workspace_bytes",
           "maskmoe_layer_backward_workspace_bytes", "maskmoe_layer_backward", "maskmoe_layer_lora_workspace_bytes",
           "maskmoe_layer_forward_lora", "maskmoe_offload_workspace_bytes", "maskmoe_offload_decode_step",
           "maskmoe_pack_expert_weights", "maskmoe_layer_forward_noalloc")
NUM_STAGES = 5
STAGES = ("route", "permute", "gate_up", "down", "combine")


class LayerDesc(ctypes.Structure):
    """``maskmoe_layer_desc``."""

    _fields_ = [(n, ctypes.c_int32) for n in
                ("T", "d", "E", "K", "F", "n_shared", "dtype", "route_mode", "gate_mode", "weight_layout")]


class Lora(ctypes.Structure):
    """``maskmoe_lora``."""

    _fields_ = [("rank", ctypes.c_int32), ("alpha", ctypes.c_float)] + [
        (n, ctypes.c_void_p) for n in ("a_gate_up", "b_gate_up", "a_down", "b_down",
                                       "as_gate_up", "bs_gate_up", "as_down", "bs_down")]


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
    lib.maskmoe_route.argtypes = [ctypes.POINTER(LayerDesc), _i32, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                  ctypes.c_size_t, _vp]
    lib.maskmoe_route.restype = ctypes.c_int
    lib.maskmoe_route_workspace_bytes.argtypes = [ctypes.POINTER(LayerDesc), _i32]
    lib.maskmoe_route_workspace_bytes.restype = ctypes.c_size_t
    lib.maskmoe_layer_workspace_bytes.argtypes = [ctypes.POINTER(LayerDesc)]
    lib.maskmoe_layer_workspace_bytes.restype = _sz
    lib.maskmoe_layer_forward.argtypes = [ctypes.POINTER(LayerDesc), _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                          _vp, _vp, _vp, _vp, _sz, _vp]
    lib.maskmoe_layer_forward.restype = ctypes.c_int
    lib.maskmoe_layer_forward_noalloc.argtypes = [ctypes.POINTER(LayerDesc), _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                                  _vp, _vp, _vp, _vp, _vp]
    lib.maskmoe_layer_forward_noalloc.restype = ctypes.c_int
    lib.maskmoe_layer_forward_profiled.argtypes = [ctypes.POINTER(LayerDesc), _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                                   _vp, _vp, _vp, _vp, _vp, _sz, _vp, _vp]
    lib.maskmoe_layer_forward_profiled.restype = ctypes.c_int
    lib.maskmoe_cache_fetches.argtypes = [_vp, _i32, _i32, _i32, _i32, _i32, _i32, _i32, _vp, _vp, _vp,
                                          _vp, _vp, _vp, _vp]
    lib.maskmoe_cache_fetches.restype = ctypes.c_int
    lib.maskmoe_status_string.argtypes = [ctypes.c_int]
    lib.maskmoe_status_string.restype = ctypes.c_char_p
    lib.maskmoe_sample_mask.argtypes = [_vp, _vp, _i32, _i32, _i32, _vp]
    lib.maskmoe_sample_mask.restype = ctypes.c_int
    lib.maskmoe_layer_forward_train.argtypes = [ctypes.POINTER(LayerDesc), _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                                _vp, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp]
    lib.maskmoe_layer_forward_train.restype = ctypes.c_int
    lib.maskmoe_stage1_backward_workspace_bytes.argtypes = [ctypes.POINTER(LayerDesc)]
    lib.maskmoe_stage1_backward_workspace_bytes.restype = _sz
    lib.maskmoe_stage1_backward.argtypes = [ctypes.POINTER(LayerDesc), _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                            _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp]
    lib.maskmoe_stage1_backward.restype = ctypes.c_int
    lib.maskmoe_layer_train_workspace_bytes.argtypes = [ctypes.POINTER(LayerDesc)]
    lib.maskmoe_layer_train_workspace_bytes.restype = _sz
    lib.maskmoe_layer_backward_workspace_bytes.argtypes = [ctypes.POINTER(LayerDesc)]
    lib.maskmoe_layer_backward_workspace_bytes.restype = _sz
    lib.maskmoe_layer_backward.argtypes = [ctypes.POINTER(LayerDesc), _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _sz,
                                           _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp]
    lib.maskmoe_layer_backward.restype = ctypes.c_int
    lib.maskmoe_layer_lora_workspace_bytes.argtypes = [ctypes.POINTER(LayerDesc)]
    lib.maskmoe_layer_lora_workspace_bytes.restype = _sz
    lib.maskmoe_layer_forward_lora.argtypes = [ctypes.POINTER(LayerDesc), _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                               ctypes.POINTER(Lora), _vp, _vp, _vp, _vp, _sz, _vp]
    lib.maskmoe_layer_forward_lora.restype = ctypes.c_int
    lib.maskmoe_offload_workspace_bytes.argtypes = [ctypes.POINTER(LayerDesc)]
    lib.maskmoe_offload_workspace_bytes.restype = _sz
    lib.maskmoe_offload_decode_step.argtypes = [ctypes.POINTER(LayerDesc), _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                                _i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp,
                                                _vp]
    lib.maskmoe_offload_decode_step.restype = ctypes.c_int
    lib.maskmoe_pack_expert_weights.argtypes = [ctypes.POINTER(LayerDesc), _i32, _vp, _vp, _vp, _vp, _vp]
    lib.maskmoe_pack_expert_weights.restype = ctypes.c_int
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


def make_desc(T, d, E, K, F=1, n_shared=0, dtype=BF16, route_mode=ROUTE_PLAIN, gate_mode=GATE_RENORM,
              weight_layout=LAYOUT_ROWS) -> LayerDesc:
    return LayerDesc(T, d, E, K, F, n_shared, dtype, route_mode, gate_mode, weight_layout)


def maskmoe_pack_expert_weights(w_gate_up=None, w_down=None):
    """Packed copies (LAYOUT_PACKED) of bf16 expert weights w_gate_up [n,2F,d] and/or
    w_down [n,d,F]; each result has its source's shape and size but the packed storage
    order, and is only meaningful to the library's entry points with weight_layout=LAYOUT_PACKED.
    Returns (packed_gate_up, packed_down), None where no source was given."""
    import torch
    if w_gate_up is None and w_down is None:
        raise ValueError("nothing to pack")
    for t, n in ((w_gate_up, "w_gate_up"), (w_down, "w_down")):
        _dev(t, n)
        if t is not None and (t.dim() != 3 or t.dtype != torch.bfloat16):
            raise ValueError(f"{n} must be a 3-d bf16 tensor")
    if w_gate_up is not None:
        n, F2, d = w_gate_up.shape
        F = F2 // 2
    else:
        n, d, F = w_down.shape
    if w_down is not None and tuple(w_down.shape) != (n, d, F):
        raise ValueError("w_down does not match w_gate_up")
    pg = torch.empty_like(w_gate_up) if w_gate_up is not None else None
    pd = torch.empty_like(w_down) if w_down is not None else None
    desc = make_desc(0, d, 1, 1, F, 0, BF16)
    _check("maskmoe_pack_expert_weights",
           load().maskmoe_pack_expert_weights(ctypes.byref(desc), n, _ptr(w_gate_up), _ptr(w_down), _ptr(pg),
                                              _ptr(pd), _stream()))
    return pg, pd


def maskmoe_route(x, w_router, K: int, route_mode: int, gate_mode: int, mask=None, prior=None,
                  with_margin: bool = True, workspace="auto"):
    """Route tokens x [T,d] through L routers w_router [L,E,d] (or [E,d] for L=1).

    mask / prior: host arrays [L,E] (or [E]). workspace: a uint8 device tensor of at least
    maskmoe_route_workspace_bytes bytes, None (selection inside the logit kernel) or "auto"
    (allocated here when the library asks for one). Returns ``(idx [L,T,K] int32,
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
    if isinstance(workspace, str):
        if workspace != "auto":
            raise ValueError("workspace: a device tensor, None or 'auto'")
        nbytes = lib.maskmoe_route_workspace_bytes(ctypes.byref(desc), L)
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=x.device) if nbytes else None
    if workspace is not None:
        _dev(workspace, "workspace")
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check("maskmoe_route", lib.maskmoe_route(ctypes.byref(desc), L, _ptr(x), _ptr(w3), m_p, p_p, _ptr(idx),
                                              _ptr(gate), _ptr(margin), _ptr(workspace), ws_bytes, _stream()))
    del m_arr, p_arr
    if squeeze:
        return idx[0], gate[0], (margin[0] if margin is not None else None)
    return idx, gate, margin


def maskmoe_layer_workspace_bytes(desc: LayerDesc) -> int:
    return int(load().maskmoe_layer_workspace_bytes(ctypes.byref(desc)))


def _forward_args(x, w_router, w_gate_up, w_down, K, route_mode, gate_mode, mask, prior, ws_gate_up, ws_down,
                  workspace, y, topk_idx, topk_gate, weight_layout=LAYOUT_ROWS, with_workspace=True):
    """Checks shapes and dtypes of a layer call and marshals its leading arguments."""
    import torch
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
    desc = make_desc(T, d, E, K, F, ns, _dtype_code(x), route_mode, gate_mode, weight_layout)
    if workspace is None and with_workspace:
        workspace = torch.empty(max(maskmoe_layer_workspace_bytes(desc), 1), dtype=torch.uint8, device=x.device)
    if y is None:
        y = torch.empty((T, d), dtype=x.dtype, device=x.device)
    m_arr, m_p = _host_u8(mask, E) if route_mode == ROUTE_HARD_MASK else (None, None)
    p_arr, p_p = _host_f32(prior, E) if route_mode == ROUTE_SOFT_PRIOR else (None, None)
    head = (ctypes.byref(desc), _ptr(x), _ptr(w_router), m_p, p_p, _ptr(w_gate_up), _ptr(w_down),
            _ptr(ws_gate_up), _ptr(ws_down), _ptr(y), _ptr(topk_idx), _ptr(topk_gate))
    return desc, workspace, y, (m_arr, p_arr), head


def maskmoe_layer_forward(x, w_router, w_gate_up, w_down, K: int, route_mode: int, gate_mode: int,
                          mask=None, prior=None, ws_gate_up=None, ws_down=None, workspace=None, y=None,
                          topk_idx=None, topk_gate=None, events=None, weight_layout=LAYOUT_ROWS):
    """One masked MoE layer. Shapes: x [T,d], w_router [E,d], w_gate_up [E,2F,d],
    w_down [E,d,F], ws_gate_up [S,2F,d], ws_down [S,d,F]; mask/prior host [E].
    ``weight_layout``: LAYOUT_PACKED when the four expert tensors come from
    maskmoe_pack_expert_weights.

    Returns y [T,d] (dtype of x). ``workspace`` (uint8 device tensor) is
    allocated when not given; ``topk_idx``/``topk_gate`` [T,K] receive the
    routing decision when given. ``events``: NUM_STAGES + 1 entries, each None or an
    already-recorded ``torch.cuda.Event(enable_timing=True)``; when given, the
    profiled entry point re-records the non-None ones around the stages.
    """
    lib = load()
    desc, workspace, y, keep, head = _forward_args(x, w_router, w_gate_up, w_down, K, route_mode, gate_mode, mask,
                                                   prior, ws_gate_up, ws_down, workspace, y, topk_idx, topk_gate,
                                                   weight_layout)
    args = head + (_ptr(workspace), workspace.numel())
    if events is None:
        _check("maskmoe_layer_forward", lib.maskmoe_layer_forward(*args, _stream()))
    else:
        if len(events) != NUM_STAGES + 1:
            raise ValueError(f"need {NUM_STAGES + 1} events")
        handles = (ctypes.c_void_p * len(events))(*[None if ev is None else ev.cuda_event for ev in events])
        _check("maskmoe_layer_forward_profiled", lib.maskmoe_layer_forward_profiled(*args, handles, _stream()))
    del keep
    return y


NOALLOC_SCRATCH_BYTES = 128 << 20


def maskmoe_layer_forward_noalloc(x, w_router, w_gate_up, w_down, K: int, route_mode: int, gate_mode: int,
                                  y, mask=None, prior=None, ws_gate_up=None, ws_down=None, topk_idx=None,
                                  topk_gate=None, weight_layout=LAYOUT_ROWS):
    """maskmoe_layer_forward with the library's own per-device scratch array as its workspace
    (the entry point for callers that cannot allocate). ``y`` [T,d] is the caller's output
    tensor; nothing is allocated here or in the library. Returns y."""
    if y is None:
        raise ValueError("maskmoe_layer_forward_noalloc writes into a caller-owned y")
    lib = load()
    _, _, y, keep, head = _forward_args(x, w_router, w_gate_up, w_down, K, route_mode, gate_mode, mask, prior,
                                        ws_gate_up, ws_down, None, y, topk_idx, topk_gate, weight_layout,
                                        with_workspace=False)
    _check("maskmoe_layer_forward_noalloc", lib.maskmoe_layer_forward_noalloc(*head, _stream()))
    del keep
    return y


def maskmoe_layer_forward_train(x, w_router, w_gate_up, w_down, K: int, route_mode: int, gate_mode: int,
                                mask=None, prior=None, ws_gate_up=None, ws_down=None, workspace=None):
    """maskmoe_layer_forward plus what the backward passes read. Returns
    ``(y [T,d], topk_idx [T,K], topk_gate [T,K], router_logits [T,E] fp32, expert_out [T,K,d] fp32)``;
    ``workspace`` (allocated with maskmoe_layer_train_workspace_bytes when not given) then holds
    what maskmoe_layer_backward reads: pass the same tensor there, unchanged."""
    import torch
    lib = load()
    T, d = x.shape
    E = w_router.shape[0]
    if workspace is None:
        F = w_gate_up.shape[1] // 2
        ns = 0 if ws_gate_up is None else ws_gate_up.shape[0]
        desc0 = make_desc(T, d, E, K, F, ns, _dtype_code(x), route_mode, gate_mode)
        workspace = torch.empty(max(int(lib.maskmoe_layer_train_workspace_bytes(ctypes.byref(desc0))), 1),
                                dtype=torch.uint8, device=x.device)
    idx = torch.empty((T, K), dtype=torch.int32, device=x.device)
    gate = torch.empty((T, K), dtype=torch.float32, device=x.device)
    logits = torch.empty((T, E), dtype=torch.float32, device=x.device)
    eo = torch.empty((T, K, d), dtype=torch.float32, device=x.device)
    desc, workspace, y, keep, head = _forward_args(x, w_router, w_gate_up, w_down, K, route_mode, gate_mode, mask,
                                                   prior, ws_gate_up, ws_down, workspace, None, idx, gate)
    _check("maskmoe_layer_forward_train",
           lib.maskmoe_layer_forward_train(*head, _ptr(logits), _ptr(eo), _ptr(workspace), workspace.numel(),
                                           _stream()))
    del keep
    return y, idx, gate, logits, eo


LORA_KEYS = ("a_gate_up", "b_gate_up", "a_down", "b_down", "as_gate_up", "bs_gate_up", "as_down", "bs_down")


def maskmoe_layer_forward_lora(x, w_router, w_gate_up, w_down, K: int, route_mode: int, gate_mode: int, lora: dict,
                               mask=None, prior=None, ws_gate_up=None, ws_down=None, workspace=None, y=None,
                               topk_idx=None, topk_gate=None, weight_layout=LAYOUT_ROWS):
    """maskmoe_layer_forward with adapted experts. ``lora``: rank, alpha and bf16 device tensors
    a_gate_up [E,2r,d], b_gate_up [E,2F,r], a_down [E,r,F], b_down [E,d,r] (and as_*/bs_* for
    the shared experts). ``workspace`` defaults to maskmoe_layer_lora_workspace_bytes bytes."""
    import torch
    lib = load()
    T, d = x.shape
    E = w_router.shape[0]
    F = w_gate_up.shape[1] // 2
    ns = 0 if ws_gate_up is None else ws_gate_up.shape[0]
    r = int(lora["rank"])
    shapes = {"a_gate_up": (E, 2 * r, d), "b_gate_up": (E, 2 * F, r), "a_down": (E, r, F), "b_down": (E, d, r),
              "as_gate_up": (ns, 2 * r, d), "bs_gate_up": (ns, 2 * F, r), "as_down": (ns, r, F),
              "bs_down": (ns, d, r)}
    for k in LORA_KEYS:
        t = lora.get(k)
        if k.startswith(("as_", "bs_")) and not ns:
            continue
        _dev(t, k)
        if t is None or tuple(t.shape) != shapes[k] or t.dtype != x.dtype or not t.is_contiguous():
            raise ValueError(f"lora[{k!r}] must be a contiguous {x.dtype} tensor of shape {shapes[k]}")
    if workspace is None:
        desc0 = make_desc(T, d, E, K, F, ns, _dtype_code(x), route_mode, gate_mode, weight_layout)
        workspace = torch.empty(max(int(lib.maskmoe_layer_lora_workspace_bytes(ctypes.byref(desc0))), 1),
                                dtype=torch.uint8, device=x.device)
    desc, workspace, y, keep, head = _forward_args(x, w_router, w_gate_up, w_down, K, route_mode, gate_mode, mask,
                                                   prior, ws_gate_up, ws_down, workspace, y, topk_idx, topk_gate,
                                                   weight_layout)
    la = Lora(r, float(lora["alpha"]), *[_ptr(lora.get(k)) if (ns or not k.startswith(("as_", "bs_"))) else None
                                         for k in LORA_KEYS])
    _check("maskmoe_layer_forward_lora",
           lib.maskmoe_layer_forward_lora(*head[:9], ctypes.byref(la), *head[9:], _ptr(workspace), workspace.numel(),
                                          _stream()))
    del keep
    return y


def offload_empty_state(E: int, B: int, device="cuda"):
    """A fresh cache state for maskmoe_offload_decode_step: int32 [B + 2E] = -1 | 0 | -1."""
    import torch
    st = torch.full((B + 2 * E,), -1, dtype=torch.int32, device=device)
    st[B:B + E] = 0
    return st


def maskmoe_offload_decode_step(x, w_router, host_w_gate_up, host_w_down, slots_gate_up, slots_down, cache_state,
                                K: int, route_mode: int, gate_mode: int, policy: int, mask=None, prior=None,
                                ws_gate_up=None, ws_down=None, counters=None, dev_error=None, workspace=None,
                                y=None, topk_idx=None, topk_gate=None, events=None, weight_layout=LAYOUT_ROWS):
    """One batch-1 decode step of one layer with host-resident experts. x [1,d] (device),
    host_w_gate_up [E,2F,d] / host_w_down [E,d,F] pinned host tensors, slots_* [B,...] device
    pool, cache_state int32 [B + 2E] device (see offload_empty_state). ``events``: 2 entries,
    each None or a torch.cuda.Event, recorded around the host-to-pool copy. Returns y [1,d]."""
    import torch
    lib = load()
    for t, n in ((x, "x"), (w_router, "w_router"), (slots_gate_up, "slots_gate_up"), (slots_down, "slots_down"),
                 (cache_state, "cache_state"), (ws_gate_up, "ws_gate_up"), (ws_down, "ws_down"),
                 (counters, "counters"), (dev_error, "dev_error"), (workspace, "workspace"), (y, "y"),
                 (topk_idx, "topk_idx"), (topk_gate, "topk_gate")):
        _dev(t, n)
    for t, n in ((host_w_gate_up, "host_w_gate_up"), (host_w_down, "host_w_down")):
        if t.is_cuda or not t.is_pinned() or not t.is_contiguous():
            raise ValueError(f"{n} must be a contiguous pinned host tensor")
    T, d = x.shape
    E, F2, d2 = host_w_gate_up.shape
    F = F2 // 2
    B = slots_gate_up.shape[0]
    if (d2 != d or tuple(host_w_down.shape) != (E, d, F) or tuple(slots_gate_up.shape) != (B, 2 * F, d)
            or tuple(slots_down.shape) != (B, d, F) or tuple(w_router.shape) != (E, d)
            or tuple(cache_state.shape) != (B + 2 * E,) or cache_state.dtype != torch.int32):
        raise ValueError("inconsistent offloaded-layer shapes")
    ns = 0 if ws_gate_up is None else ws_gate_up.shape[0]
    desc = make_desc(T, d, E, K, F, ns, _dtype_code(x), route_mode, gate_mode, weight_layout)
    if workspace is None:
        workspace = torch.empty(max(int(lib.maskmoe_offload_workspace_bytes(ctypes.byref(desc))), 1),
                                dtype=torch.uint8, device=x.device)
    if y is None:
        y = torch.empty((T, d), dtype=x.dtype, device=x.device)
    m_arr, m_p = _host_u8(mask, E) if route_mode == ROUTE_HARD_MASK else (None, None)
    p_arr, p_p = _host_f32(prior, E) if route_mode == ROUTE_SOFT_PRIOR else (None, None)
    handles = None
    if events is not None:
        if len(events) != 2:
            raise ValueError("events needs 2 entries")
        handles = (ctypes.c_void_p * 2)(*[None if ev is None else ev.cuda_event for ev in events])
    _check("maskmoe_offload_decode_step",
           lib.maskmoe_offload_decode_step(ctypes.byref(desc), _ptr(x), _ptr(w_router), m_p, p_p,
                                           _ptr(host_w_gate_up), _ptr(host_w_down), _ptr(ws_gate_up),
                                           _ptr(ws_down), B, policy, _ptr(slots_gate_up), _ptr(slots_down),
                                           _ptr(cache_state), _ptr(y), _ptr(topk_idx), _ptr(topk_gate),
                                           _ptr(counters), _ptr(dev_error), _ptr(workspace), workspace.numel(),
                                           handles, _stream()))
    del m_arr, p_arr
    return y


def maskmoe_sample_mask(mask_logits, uniforms, e_keep: int) -> np.ndarray:
    """Binary masks [L,E] (or [E]) with e_keep ones, drawn without replacement from
    softmax(mask_logits) using the given uniforms [L,e_keep] (or [e_keep]) in [0, 1)."""
    lib = load()
    ml = np.ascontiguousarray(np.asarray(mask_logits, dtype=np.float32))
    squeeze = ml.ndim == 1
    ml2 = ml.reshape(1, -1) if squeeze else ml
    L, E = ml2.shape
    u = np.ascontiguousarray(np.asarray(uniforms, dtype=np.float64).reshape(L, e_keep))
    out = np.zeros((L, E), dtype=np.uint8)
    _check("maskmoe_sample_mask", lib.maskmoe_sample_mask(ml2.ctypes.data_as(ctypes.c_void_p),
                                                          u.ctypes.data_as(ctypes.c_void_p), L, E, e_keep,
                                                          out.ctypes.data_as(ctypes.c_void_p)))
    return out[0] if squeeze else out


def maskmoe_stage1_backward(x, w_router, K: int, gate_mode: int, mask, topk_idx, router_logits, dy, expert_out,
                            mask_logits=None, d_mask_logits=None, with_d_x: bool = True, workspace=None):
    """Mask and router gradients of one hard-mask step (Eq. 2, Eq. 3). ``d_mask_logits`` (fp32
    device [E]) is accumulated in place when given (mask_logits host [E] then required).
    Returns dict(d_gate [T,K], d_mask [E], d_w_router [E,d], d_x [T,d] or None), fp32."""
    import torch
    lib = load()
    for t, n in ((x, "x"), (w_router, "w_router"), (topk_idx, "topk_idx"), (router_logits, "router_logits"),
                 (dy, "dy"), (expert_out, "expert_out"), (d_mask_logits, "d_mask_logits"),
                 (workspace, "workspace")):
        _dev(t, n)
    T, d = x.shape
    E = w_router.shape[0]
    if tuple(w_router.shape) != (E, d) or tuple(dy.shape) != (T, d) or tuple(expert_out.shape) != (T, K, d) \
            or tuple(topk_idx.shape) != (T, K) or tuple(router_logits.shape) != (T, E):
        raise ValueError("inconsistent shapes")
    if w_router.dtype != x.dtype or dy.dtype != x.dtype:
        raise ValueError("x, w_router and dy must share a dtype")
    if expert_out.dtype != torch.float32 or router_logits.dtype != torch.float32 or topk_idx.dtype != torch.int32:
        raise ValueError("expert_out and router_logits are float32, topk_idx int32")
    desc = make_desc(T, d, E, K, 1, 0, _dtype_code(x), ROUTE_HARD_MASK, gate_mode)
    need = int(lib.maskmoe_stage1_backward_workspace_bytes(ctypes.byref(desc)))
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
    m_arr, m_p = _host_u8(mask, E)
    ml_arr, ml_p = _host_f32(mask_logits, E)
    out = dict(d_gate=torch.empty((T, K), dtype=torch.float32, device=x.device),
               d_mask=torch.empty(E, dtype=torch.float32, device=x.device),
               d_w_router=torch.empty((E, d), dtype=torch.float32, device=x.device),
               d_x=torch.empty((T, d), dtype=torch.float32, device=x.device) if with_d_x else None)
    _check("maskmoe_stage1_backward",
           lib.maskmoe_stage1_backward(ctypes.byref(desc), _ptr(x), _ptr(w_router), m_p, ml_p, _ptr(topk_idx),
                                       _ptr(router_logits), _ptr(dy), _ptr(expert_out), _ptr(out["d_gate"]),
                                       _ptr(out["d_mask"]), _ptr(d_mask_logits), _ptr(out["d_w_router"]),
                                       _ptr(out["d_x"]), _ptr(workspace), workspace.numel(), _stream()))
    del m_arr, ml_arr
    return out


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


def maskmoe_layer_backward(x, w_gate_up, w_down, K: int, gate_mode: int, topk_gate, dy, train_workspace,
                           ws_gate_up=None, ws_down=None, route_mode: int = ROUTE_HARD_MASK, workspace=None):
    """Experts' side of the layer backward (bf16). ``train_workspace`` is the workspace of the
    maskmoe_layer_forward_train call with the same arguments. Returns dict(d_x [T,d],
    d_w_gate_up [E,2F,d], d_w_down [E,d,F], d_ws_gate_up, d_ws_down), fp32."""
    import torch
    lib = load()
    for t, n in ((x, "x"), (w_gate_up, "w_gate_up"), (w_down, "w_down"), (ws_gate_up, "ws_gate_up"),
                 (ws_down, "ws_down"), (topk_gate, "topk_gate"), (dy, "dy"), (train_workspace, "train_workspace"),
                 (workspace, "workspace")):
        _dev(t, n)
    T, d = x.shape
    E, F2, _ = w_gate_up.shape
    F = F2 // 2
    ns = 0 if ws_gate_up is None else ws_gate_up.shape[0]
    if tuple(dy.shape) != (T, d) or tuple(topk_gate.shape) != (T, K) or tuple(w_down.shape) != (E, d, F):
        raise ValueError("inconsistent shapes")
    desc = make_desc(T, d, E, K, F, ns, _dtype_code(x), route_mode, gate_mode)
    need = int(lib.maskmoe_layer_backward_workspace_bytes(ctypes.byref(desc)))
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
    f32 = dict(dtype=torch.float32, device=x.device)
    out = dict(d_x=torch.empty((T, d), **f32), d_w_gate_up=torch.empty((E, F2, d), **f32),
               d_w_down=torch.empty((E, d, F), **f32),
               d_ws_gate_up=torch.empty((ns, F2, d), **f32) if ns else None,
               d_ws_down=torch.empty((ns, d, F), **f32) if ns else None)
    _check("maskmoe_layer_backward",
           lib.maskmoe_layer_backward(ctypes.byref(desc), _ptr(x), _ptr(w_gate_up), _ptr(w_down), _ptr(ws_gate_up),
                                      _ptr(ws_down), _ptr(topk_gate), _ptr(dy), _ptr(train_workspace),
                                      train_workspace.numel(), _ptr(out["d_x"]), _ptr(out["d_w_gate_up"]),
                                      _ptr(out["d_w_down"]), _ptr(out["d_ws_gate_up"]), _ptr(out["d_ws_down"]),
                                      _ptr(workspace), workspace.numel(), _stream()))
    return out
