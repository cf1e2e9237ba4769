"""Oracle: expert FFN and gate-weighted combine (float64). Test infrastructure only.

The layer output of Eq. 1 (Section 3.1) is y = sum_{i in A} g_i F_i(x), plus
the outputs of the shared experts, which see every token and are added with
weight 1 (Section 3.1, on DeepSeek-V2-Lite). The paper leaves the expert
F_i abstract; the SwiGLU form of the Mixtral and DeepSeek experts is taken:
F(x) = W_down (SiLU(W_gate x) * (W_up x)), no biases, SiLU(u) = u/(1+e^-u).

Weight layout: ``w_gate_up [E, 2F, d]`` with gate rows 0..F-1 and up rows
F..2F-1; ``w_down [E, d, F]``. Weights may be passed in their stored form
together with a ``widen`` callable that returns exact float64 values; the
oracle widens one expert at a time so that large layers fit in memory.
Everything is computed in float64 with no intermediate rounding.

Stage 2 (Section 3.2; Section 4 setup and Appendix B) fine-tunes the experts with low-rank
adapters: every routed expert, and the shared experts, of rank r = 8 and alpha = 16. An
adapted projection W (out x in) acts as W x + (alpha / r) B (A x) with A [r, in] and
B [out, r] (``lora_expert_ffn``, ``lora_moe_layer``); the paper does not list the adapted
projections, and the gate, up and down projections of each expert are taken.
"""

from __future__ import annotations

from typing import Callable, Optional

import numpy as np


def _f64(a):
    return np.asarray(a, dtype=np.float64)


def silu(u: np.ndarray) -> np.ndarray:
    """SiLU(u) = u / (1 + exp(-u))."""
    return u / (1.0 + np.exp(-u))


def expert_ffn(x: np.ndarray, w_gate_up: np.ndarray, w_down: np.ndarray) -> np.ndarray:
    """F(x) = W_down (SiLU(W_gate x) * W_up x) for rows x [n,d]; one expert's float64 weights."""
    F = w_down.shape[1]
    g = x @ w_gate_up[:F].T
    u = x @ w_gate_up[F:].T
    return (silu(g) * u) @ w_down.T


def moe_layer(x, idx, gate, w_gate_up, w_down, ws_gate_up=None, ws_down=None,
              widen: Optional[Callable] = None) -> np.ndarray:
    """y_t = sum_k gate[t,k] * F_{idx[t,k]}(x_t) + sum_s F_s(x_t)  (Eq. 1; shared experts of Section 3.1).

    x [T,d] (float64), idx/gate [T,K]. Each expert is evaluated on exactly
    the tokens that selected it; ``widen`` maps a stored weight tensor to
    float64 (identity when None).
    """
    wd = widen if widen is not None else _f64
    x = _f64(x)
    idx = np.asarray(idx)
    gate = _f64(gate)
    T, d = x.shape
    y = np.zeros((T, d), dtype=np.float64)
    E = w_gate_up.shape[0]
    for e in range(E):
        rows, slots = np.nonzero(idx == e)
        if rows.size == 0:
            continue
        out = expert_ffn(x[rows], wd(w_gate_up[e]), wd(w_down[e]))
        np.add.at(y, rows, gate[rows, slots][:, None] * out)
    if ws_gate_up is not None:
        for s in range(ws_gate_up.shape[0]):
            y += expert_ffn(x, wd(ws_gate_up[s]), wd(ws_down[s]))
    return y


def moe_token(x_t, idx_t, gate_t, w_gate_up, w_down, ws_gate_up=None, ws_down=None,
              widen: Optional[Callable] = None) -> np.ndarray:
    """Output of a single token (the same definition, evaluated one token at a time)."""
    return moe_layer(_f64(x_t)[None, :], np.asarray(idx_t)[None, :], _f64(gate_t)[None, :],
                     w_gate_up, w_down, ws_gate_up, ws_down, widen)[0]


def lora_linear(x, w, a, b, scale: float) -> np.ndarray:
    """x W^T + scale (x A^T) B^T: an adapted projection, rows x [n, in], W [out, in], A [r, in],
    B [out, r]."""
    x = _f64(x)
    return x @ _f64(w).T + scale * ((x @ _f64(a).T) @ _f64(b).T)


def lora_expert_ffn(x, w_gate_up, w_down, a_gate_up, b_gate_up, a_down, b_down, scale: float) -> np.ndarray:
    """SwiGLU expert with adapted gate, up and down projections. Adapter layout: a_gate_up
    [2r, d] (A_gate rows, then A_up rows), b_gate_up [2F, r] (B_gate rows, then B_up rows),
    a_down [r, F], b_down [d, r]."""
    F = w_down.shape[1]
    r = a_down.shape[0]
    g = lora_linear(x, w_gate_up[:F], a_gate_up[:r], b_gate_up[:F], scale)
    u = lora_linear(x, w_gate_up[F:], a_gate_up[r:], b_gate_up[F:], scale)
    return lora_linear(silu(g) * u, w_down, a_down, b_down, scale)


def lora_moe_layer(x, idx, gate, w_gate_up, w_down, lora, ws_gate_up=None, ws_down=None,
                   widen: Optional[Callable] = None) -> np.ndarray:
    """Eq. 1 with adapted experts. ``lora`` is a dict: rank, alpha, a_gate_up [E,2r,d],
    b_gate_up [E,2F,r], a_down [E,r,F], b_down [E,d,r] and, with shared experts,
    as_gate_up, bs_gate_up, as_down, bs_down [S, ...]."""
    wd = widen if widen is not None else _f64
    scale = float(lora["alpha"]) / float(lora["rank"])
    x = _f64(x)
    idx = np.asarray(idx)
    gate = _f64(gate)
    T, d = x.shape
    y = np.zeros((T, d), dtype=np.float64)
    for e in range(w_gate_up.shape[0]):
        rows, slots = np.nonzero(idx == e)
        if rows.size == 0:
            continue
        out = lora_expert_ffn(x[rows], wd(w_gate_up[e]), wd(w_down[e]), wd(lora["a_gate_up"][e]),
                              wd(lora["b_gate_up"][e]), wd(lora["a_down"][e]), wd(lora["b_down"][e]), scale)
        np.add.at(y, rows, gate[rows, slots][:, None] * out)
    if ws_gate_up is not None:
        for s_ in range(ws_gate_up.shape[0]):
            y += lora_expert_ffn(x, wd(ws_gate_up[s_]), wd(ws_down[s_]), wd(lora["as_gate_up"][s_]),
                                 wd(lora["bs_gate_up"][s_]), wd(lora["as_down"][s_]), wd(lora["bs_down"][s_]), scale)
    return y
