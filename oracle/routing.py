"""Oracle: routing of the masked MoE layer (float64). Test infrastructure only.

Follows Section 3.1 (router logits, softmax, Top-K, gate rules: Eq. 1),
Section 3.2 Stage 1 (hard binary mask, Eq. 2, and the gate values under it)
and Section 3.2 Evaluation and inference (soft prior re-ranking, Eq. 4,
gates from p).

Readings where the paper is silent:
* ties in Top-K go to the lower expert index; the selected experts are
  listed by decreasing key, then increasing index;
* ranking is done on log-domain keys (z_i, or z_i + log pi_i), which order
  the experts exactly as the products p_i*m_i and p_i*pi_i of Eq. 2 and
  Eq. 4 do (softmax is monotone and shares its normaliser), without the
  underflow of exp; masked experts get key -inf and are never eligible;
* the margin of a token is the gap, in logit units, between its K-th and
  (K+1)-th log-domain keys (+inf when fewer than K+1 experts are eligible).
"""

from __future__ import annotations

import numpy as np

PLAIN, HARD_MASK, SOFT_PRIOR = 0, 1, 2
GATE_P, GATE_RENORM = 0, 1


def router_logits(x: np.ndarray, w: np.ndarray) -> np.ndarray:
    """z = W x for every token (Section 3.1). x [T,d], W [E,d] -> z [T,E], float64."""
    return np.asarray(x, dtype=np.float64) @ np.asarray(w, dtype=np.float64).T


def softmax(z: np.ndarray) -> np.ndarray:
    """p = softmax(z) over the last axis (Section 3.1), float64."""
    z = np.asarray(z, dtype=np.float64)
    e = np.exp(z - z.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def literal_keys(p: np.ndarray, mode: int, mask=None, prior=None) -> np.ndarray:
    """The selection keys as the paper writes them: p (Eq. 1), p*m (Eq. 2), p*pi (Eq. 4)."""
    if mode == PLAIN:
        return p.copy()
    if mode == HARD_MASK:
        return p * np.asarray(mask, dtype=np.float64)
    if mode == SOFT_PRIOR:
        return p * np.asarray(prior, dtype=np.float64)
    raise ValueError(f"unknown route mode {mode}")


def log_keys(z: np.ndarray, mode: int, mask=None, prior=None) -> np.ndarray:
    """Log-domain keys that order experts as ``literal_keys`` does (up to a per-token constant).

    plain: z_i; hard mask: z_i where m_i = 1, -inf where m_i = 0;
    soft prior: z_i + log pi_i.
    """
    z = np.asarray(z, dtype=np.float64)
    if mode == PLAIN:
        return z.copy()
    if mode == HARD_MASK:
        m = np.asarray(mask).astype(bool)
        return np.where(m, z, -np.inf)
    if mode == SOFT_PRIOR:
        return z + np.log(np.asarray(prior, dtype=np.float64))
    raise ValueError(f"unknown route mode {mode}")


def top_k(keys: np.ndarray, K: int):
    """Indices of the K largest keys per row, ordered by (-key, index); and the K-th/(K+1)-th gap.

    A stable sort of -key keeps equal keys in index order, which is the
    lower-index tie rule.
    """
    keys = np.asarray(keys, dtype=np.float64)
    order = np.argsort(-keys, axis=-1, kind="stable")
    idx = order[..., :K]
    srt = np.take_along_axis(keys, order, axis=-1)
    kth = srt[..., K - 1]
    if keys.shape[-1] > K:
        nxt = srt[..., K]
        with np.errstate(invalid="ignore"):
            margin = np.where(np.isneginf(nxt), np.inf, kth - nxt)
    else:
        margin = np.full(kth.shape, np.inf)
    return idx.astype(np.int64), margin


def gates(p: np.ndarray, idx: np.ndarray, gate_mode: int) -> np.ndarray:
    """Gate values of the selected experts, always from the full softmax p (Section 3.1).

    GATE_P: g_i = p_i (DeepSeek-V2-Lite). GATE_RENORM: g_i = p_i / sum_{j in A} p_j
    (Mixtral-8x7B). Under the hard mask the values computed from p*m equal
    these on the active set (Section 3.2, Stage 1); under the prior the gates
    stay those of p (Section 3.2, Evaluation and inference).
    """
    sel = np.take_along_axis(p, idx, axis=-1)
    if gate_mode == GATE_P:
        return sel
    if gate_mode == GATE_RENORM:
        return sel / sel.sum(axis=-1, keepdims=True)
    raise ValueError(f"unknown gate mode {gate_mode}")


def route_logits(z: np.ndarray, K: int, mode: int, gate_mode: int, mask=None, prior=None):
    """Routing of tokens given their router logits z [T,E].

    Returns ``(idx [T,K] int64, gate [T,K] float64, margin [T] float64)``.
    """
    z = np.asarray(z, dtype=np.float64)
    p = softmax(z)
    idx, margin = top_k(log_keys(z, mode, mask, prior), K)
    return idx, gates(p, idx, gate_mode), margin


def route(x, w, K: int, mode: int, gate_mode: int, mask=None, prior=None):
    """Routing of tokens x [T,d] through router W [E,d]: Eq. 1 / Eq. 2 / Eq. 4 by ``mode``."""
    return route_logits(router_logits(x, w), K, mode, gate_mode, mask, prior)


def route_layers(x, w_layers, K: int, mode: int, gate_mode: int, masks=None, priors=None):
    """Routing of the same tokens through L independent routers W [L,E,d] (one mask/prior per layer).

    Returns ``idx [L,T,K]``, ``gate [L,T,K]``, ``margin [L,T]``.
    """
    L = len(w_layers)
    res = [route(x, w_layers[l], K, mode, gate_mode,
                 None if masks is None else masks[l],
                 None if priors is None else priors[l]) for l in range(L)]
    return (np.stack([r[0] for r in res]), np.stack([r[1] for r in res]),
            np.stack([r[2] for r in res]))


def valid_selection(z_row: np.ndarray, chosen, K: int, mode: int, mask=None, prior=None,
                    tol: float = 1e-3) -> bool:
    """Whether a selected set is a correct Top-K up to ``tol`` logit units.

    Every chosen expert must be eligible, distinct, and have a log-domain key
    no smaller than the K-th largest key minus ``tol``. Used where several
    answers are correct (near-ties).
    """
    chosen = [int(c) for c in chosen]
    if len(chosen) != K or len(set(chosen)) != K:
        return False
    lk = log_keys(np.asarray(z_row, dtype=np.float64)[None, :], mode,
                  None if mask is None else np.asarray(mask)[None, :],
                  None if prior is None else np.asarray(prior)[None, :])[0]
    kth = np.sort(lk)[::-1][K - 1]
    return all(np.isfinite(lk[c]) and lk[c] >= kth - tol for c in chosen)
