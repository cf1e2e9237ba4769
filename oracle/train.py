"""Oracle: Stage 1 of masked co-adaptive fine-tuning, the mask and router gradients (float64).
Test infrastructure only.

Section 3.2, Stage 1 (Eq. 2): pi = softmax(m~) over the real-valued mask m~; E' distinct
experts are drawn from pi by multinomial sampling without replacement and form the binary
mask m; A = Top-K(p * m) and the gate weights are computed from p * m (on A they equal those
computed from p, since m = 1 there). All tokens of a batch share the mask.

Section 3.2, Mask optimization (Eq. 3): the loss reaches m through the gate weights of the
active experts, so dL/dm sums every token's contribution; the straight-through estimator
takes dL/dpi = dL/dm, and the softmax Jacobian gives dL/dm~ = (diag(pi) - pi pi^T) dL/dm.
The gradient of m~ is accumulated over T steps before one update (Stage 1; T = 1 for
Mixtral, 100 for DeepSeek-V2-Lite in Appendix B).

Eq. 1 gives y_t = sum_{i in A_t} g_i F_i(x_t) (+ shared experts), so for a cotangent dy the
gate cotangent is dL/dg_{t,i} = <dy_t, F_i(x_t)>; the router is z = W x, p = softmax(z).
The experts are fine-tuned too (the routers and experts update at every step, Stage 1; Stage 2
continues with them): with the gates held fixed, expert i receives dL/dF_i(x_t) = g_i dy_t,
and the chain rule through its SwiGLU F(x) = W_down (SiLU(W_gate x) * W_up x) gives its
weight gradients and its share of dL/dx (``expert_backward``, ``moe_layer_backward``).

Readings where the paper is silent:
* the sampler draws one expert per uniform u in [0, 1): among the experts not yet drawn, in
  increasing index order, the first whose running sum of pi exceeds u times their total;
  the caller supplies the uniforms;
* "gate weights computed from p * m" with m a real vector means g_i = p_i m_i (gate rule
  g = p) or g_i = p_i m_i / sum_{j in A} p_j m_j (renormalised rule), the set A held fixed:
  the gradient is that of the gate values, not of the discrete Top-K choice.
"""

from __future__ import annotations

import numpy as np

from . import routing as R


def mask_distribution(mask_logits) -> np.ndarray:
    """pi = softmax(m~) (Eq. 2), float64."""
    return R.softmax(np.asarray(mask_logits, dtype=np.float64))


def sample_mask(mask_logits, uniforms, e_keep: int) -> np.ndarray:
    """Binary mask with exactly e_keep ones: successive draws without replacement from pi
    (Eq. 2), draw s using uniforms[s] by inverse CDF over the remaining experts."""
    pi = mask_distribution(mask_logits)
    E = pi.shape[0]
    if not 1 <= e_keep <= E:
        raise ValueError("need 1 <= E' <= E")
    remaining = list(range(E))
    mask = np.zeros(E, dtype=np.uint8)
    for s in range(e_keep):
        total = 0.0
        for i in remaining:
            total += pi[i]
        target = float(uniforms[s]) * total
        run = 0.0
        pick = remaining[-1]          # u * total below the full sum always lands earlier
        for i in remaining:
            run += pi[i]
            if target < run:
                pick = i
                break
        mask[pick] = 1
        remaining.remove(pick)
    return mask


def inclusion_probabilities(mask_logits, e_keep: int) -> np.ndarray:
    """Exact probability that each expert is in the sampled set, by enumerating every ordered
    sequence of e_keep distinct draws: P(i_1..i_s) = prod_s pi_{i_s} / (1 - sum_{r<s} pi_{i_r}).
    Small E only (the count of sequences is E! / (E - e_keep)!)."""
    pi = mask_distribution(mask_logits)
    E = pi.shape[0]
    inc = np.zeros(E)

    def walk(prefix, prob, used):
        if len(prefix) == e_keep:
            inc[list(prefix)] += prob
            return
        left = 1.0 - used
        for i in range(E):
            if i not in prefix:
                walk(prefix + (i,), prob * pi[i] / left, used + pi[i])

    walk((), 1.0, 0.0)
    return inc


def gate_cotangent(dy, expert_out) -> np.ndarray:
    """dL/dg_{t,k} = <dy_t, F_{A_t[k]}(x_t)> (Eq. 1). dy [T,d], expert_out [T,K,d] -> [T,K]."""
    dy = np.asarray(dy, dtype=np.float64)
    eo = np.asarray(expert_out, dtype=np.float64)
    return np.einsum("td,tkd->tk", dy, eo)


def mask_router_grad(z, idx, dg, gate_mode: int, mask):
    """Gradients of the gate values of Eq. 2 with respect to the mask and the router logits.

    z [T,E] router logits, idx [T,K] the active sets, dg [T,K] gate cotangents, mask [E]
    the binary mask (1 on every active expert). The gate Jacobians are written out as
    matrices over the active set; the softmax Jacobian carries dL/dp to dL/dz.
    Returns (d_mask [E] summed over tokens, dz [T,E]).
    """
    z = np.asarray(z, dtype=np.float64)
    p = R.softmax(z)
    m = np.asarray(mask, dtype=np.float64)
    T, E = z.shape
    d_mask = np.zeros(E)
    dz = np.zeros((T, E))
    for t in range(T):
        A = np.asarray(idx[t], dtype=np.int64)
        pa, ma, dga = p[t, A], m[A], np.asarray(dg[t], dtype=np.float64)
        if gate_mode == R.GATE_P:                     # g_i = p_i m_i
            jac_m = np.diag(pa)                       # dg_i / dm_k
            jac_p = np.diag(ma)                       # dg_i / dp_k
        elif gate_mode == R.GATE_RENORM:              # g_i = p_i m_i / S, S = sum_A p_j m_j
            S = float(np.sum(pa * ma))
            jac_m = (np.diag(pa) * S - np.outer(pa * ma, pa)) / S ** 2
            jac_p = (np.diag(ma) * S - np.outer(pa * ma, ma)) / S ** 2
        else:
            raise ValueError(f"unknown gate mode {gate_mode}")
        np.add.at(d_mask, A, dga @ jac_m)
        dp = np.zeros(E)
        dp[A] = dga @ jac_p
        dz[t] = (np.diag(p[t]) - np.outer(p[t], p[t])) @ dp
    return d_mask, dz


def router_weight_grad(dz, x) -> np.ndarray:
    """dL/dW = dz^T x for z = W x. dz [T,E], x [T,d] -> [E,d]."""
    return np.asarray(dz, dtype=np.float64).T @ np.asarray(x, dtype=np.float64)


def router_input_grad(dz, w) -> np.ndarray:
    """The router's share of dL/dx: dz W. dz [T,E], W [E,d] -> [T,d]."""
    return np.asarray(dz, dtype=np.float64) @ np.asarray(w, dtype=np.float64)


def ste_mask_logits_grad(d_mask, mask_logits) -> np.ndarray:
    """Eq. 3: dL/dm~ = (diag(pi) - pi pi^T) dL/dm, pi = softmax(m~)."""
    pi = mask_distribution(mask_logits)
    return (np.diag(pi) - np.outer(pi, pi)) @ np.asarray(d_mask, dtype=np.float64)


def stage1_backward(x, w_router, mask, mask_logits, idx, dy, expert_out, gate_mode: int):
    """One step's mask and router gradients for a hard-mask layer (Eq. 2, Eq. 3).

    Returns dict(dg [T,K], d_mask [E], d_mask_logits [E], dz [T,E], d_w_router [E,d],
    d_x_router [T,d]).
    """
    z = R.router_logits(x, w_router)
    dg = gate_cotangent(dy, expert_out)
    d_mask, dz = mask_router_grad(z, idx, dg, gate_mode, mask)
    return dict(dg=dg, d_mask=d_mask, d_mask_logits=ste_mask_logits_grad(d_mask, mask_logits), dz=dz,
                d_w_router=router_weight_grad(dz, x), d_x_router=router_input_grad(dz, w_router))


def silu_grad(a):
    """d SiLU(a) / da = s (1 + a (1 - s)), s = 1 / (1 + e^-a)."""
    a = np.asarray(a, dtype=np.float64)
    s = 1.0 / (1.0 + np.exp(-a))
    return s * (1.0 + a * (1.0 - s))


def expert_backward(x, dout, w_gate_up, w_down):
    """Gradients of sum_r <dout_r, F(x_r)> for one SwiGLU expert on rows x [n,d].

    a = x W_gate^T, b = x W_up^T, h = SiLU(a) * b, F = h W_down^T; then
    dh = dout W_down, dW_down = dout^T h, da = dh * b * SiLU'(a), db = dh * SiLU(a),
    dx = da W_gate + db W_up, dW_gate = da^T x, dW_up = db^T x.
    Returns (dx [n,d], dW_gate_up [2F,d], dW_down [d,F]), float64.
    """
    x = np.asarray(x, dtype=np.float64)
    dout = np.asarray(dout, dtype=np.float64)
    wgu = np.asarray(w_gate_up, dtype=np.float64)
    wd = np.asarray(w_down, dtype=np.float64)
    F = wd.shape[1]
    wg, wu = wgu[:F], wgu[F:]
    a = x @ wg.T
    b = x @ wu.T
    sa = a / (1.0 + np.exp(-a))
    h = sa * b
    dh = dout @ wd
    d_wd = dout.T @ h
    da = dh * b * silu_grad(a)
    db = dh * sa
    dx = da @ wg + db @ wu
    return dx, np.concatenate([da.T @ x, db.T @ x], axis=0), d_wd


def moe_layer_backward(x, idx, gate, dy, w_gate_up, w_down, ws_gate_up=None, ws_down=None, widen=None):
    """Expert-side gradients of L = sum_t <dy_t, y_t> for the layer of Eq. 1 with the routing
    (idx, gate) held fixed: routed expert e gets dout = gate * dy on the tokens that chose it,
    a shared expert dout = dy on every token.

    Returns dict(dx [T,d] (the experts' share of dL/dx), d_w_gate_up [E,2F,d], d_w_down [E,d,F],
    d_ws_gate_up, d_ws_down (None without shared experts)), float64.
    """
    wdn = widen if widen is not None else (lambda a: np.asarray(a, dtype=np.float64))
    x = np.asarray(x, dtype=np.float64)
    dy = np.asarray(dy, dtype=np.float64)
    idx = np.asarray(idx)
    gate = np.asarray(gate, dtype=np.float64)
    T, d = x.shape
    E, F2, _ = w_gate_up.shape
    F = F2 // 2
    dx = np.zeros((T, d))
    d_wgu = np.zeros((E, F2, d))
    d_wd = np.zeros((E, d, F))
    for e in range(E):
        rows, slots = np.nonzero(idx == e)
        if rows.size == 0:
            continue
        dout = gate[rows, slots][:, None] * dy[rows]
        gx, d_wgu[e], d_wd[e] = expert_backward(x[rows], dout, wdn(w_gate_up[e]), wdn(w_down[e]))
        np.add.at(dx, rows, gx)
    out = dict(dx=dx, d_w_gate_up=d_wgu, d_w_down=d_wd, d_ws_gate_up=None, d_ws_down=None)
    if ws_gate_up is not None:
        S = ws_gate_up.shape[0]
        out["d_ws_gate_up"] = np.zeros((S, F2, d))
        out["d_ws_down"] = np.zeros((S, d, F))
        for s in range(S):
            gx, out["d_ws_gate_up"][s], out["d_ws_down"][s] = expert_backward(x, dy, wdn(ws_gate_up[s]),
                                                                              wdn(ws_down[s]))
            dx += gx
    return out
