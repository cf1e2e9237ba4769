"""Helpers of the GPU parity tests: device upload of synthetic inputs and the comparison
rules against the oracle.

Routing parity rule: where the oracle's margin (gap between the K-th and (K+1)-th
log-domain keys) exceeds 1e-3 logit units the selected expert sets must be identical;
elsewhere several answers are correct and the GPU's set must be a valid Top-K within
1e-3 of the K-th key. Gates are compared per selected expert for every token: with the
oracle's gates where the sets must match, and at near-ties with the gates the oracle computes
from its own softmax p on the GPU's (validated) set (Section 3.1's gate rule). The oracle's
FFN and cache replay then run on that same effective routing (``effective_routing``), so no
token is left out of any output comparison. Output parity:
max |y_gpu - y_ref| / max |y_ref| <= 1e-2 for bf16 (fp32 accumulation, H rounded to bf16,
one final bf16 rounding) and <= 2e-5 for fp32.
"""

import sys

import numpy as np
import torch

from oracle import routing as R
from paper_2609_34077_amd import synth

MARGIN_TOL = 1e-3
BF16_TOL = 1e-2
F32_TOL = 2e-5


def say(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def dev(a: np.ndarray, dtype: str = None) -> torch.Tensor:
    """Upload a stored array: uint16 bf16 bits -> bfloat16, float32 -> float32, ints as is."""
    t = torch.from_numpy(np.ascontiguousarray(a))
    if a.dtype == np.uint16:
        t = t.view(torch.bfloat16)
    return t.cuda()


def f64(a: np.ndarray, dtype: str) -> np.ndarray:
    return synth.widen(a, dtype)


def check_routing(z, idx_g, gate_g, margin_g, K, mode, gate_mode, mask=None, prior=None,
                  gate_rtol=2e-5, margin_atol=2e-4):
    """Compare GPU routing [T,K] with the oracle routing of logits z [T,E] (float64).

    Returns the number of near-tie tokens (oracle margin <= 1e-3).
    """
    idx_o, gate_o, margin_o = R.route_logits(z, K, mode, gate_mode, mask, prior)
    idx_g = np.asarray(idx_g)
    gate_g = np.asarray(gate_g, dtype=np.float64)
    T = z.shape[0]
    near = 0
    p = R.softmax(z)
    for t in range(T):
        if margin_o[t] > MARGIN_TOL:
            if set(idx_g[t].tolist()) != set(idx_o[t].tolist()):
                raise AssertionError(f"token {t}: gpu {idx_g[t]} oracle {idx_o[t]} margin {margin_o[t]}")
            go = dict(zip(idx_o[t].tolist(), gate_o[t].tolist()))
        else:
            near += 1
            assert R.valid_selection(z[t], idx_g[t], K, mode, mask, prior, MARGIN_TOL), (t, idx_g[t])
            # the oracle's gates on the GPU's set: Section 3.1's rule applied to the oracle's p
            go = dict(zip(idx_g[t].tolist(), R.gates(p[t:t + 1], idx_g[t:t + 1].astype(np.int64),
                                                     gate_mode)[0].tolist()))
        for j, e in enumerate(idx_g[t].tolist()):
            assert abs(gate_g[t, j] - go[e]) <= gate_rtol * max(abs(go[e]), 1e-30) + 1e-7, (t, e)
    if margin_g is not None:
        mg = np.asarray(margin_g, dtype=np.float64)
        fin = np.isfinite(margin_o)
        assert (np.isinf(mg) == ~fin).all()
        assert np.abs(mg[fin] - margin_o[fin]).max(initial=0.0) <= margin_atol
    return near


def effective_routing(z, idx_g, K, mode, gate_mode, mask=None, prior=None):
    """The routing the oracle's FFN and cache replay run on (the near-tie reading of the routing
    parity rule): the oracle's own sets and gates where its margin exceeds 1e-3; at near-ties the
    GPU's set, after checking that it is a valid Top-K, with gates from the oracle's softmax p.

    Returns ``(idx [T,K] int64, gate [T,K] float64, near [T] bool)``.
    """
    idx_o, gate_o, margin_o = R.route_logits(z, K, mode, gate_mode, mask, prior)
    idx_g = np.asarray(idx_g).astype(np.int64)
    near = ~(margin_o > MARGIN_TOL)
    for t in np.flatnonzero(near):
        assert R.valid_selection(z[t], idx_g[t], K, mode, mask, prior, MARGIN_TOL), (t, idx_g[t])
    idx = np.where(near[:, None], idx_g, idx_o)
    gate = np.where(near[:, None], R.gates(R.softmax(z), idx, gate_mode), gate_o)
    return idx, gate, near


def tile_sample_tokens(idx_g, E, n_shared=0, tile=256, seed=0, per_tile=3):
    """Tokens whose outputs cover every 256-row tile of every expert group of the grouped GEMMs.

    The permutation lays out group e as the (token, slot) pairs that chose e, in pair order
    (t * K + k), and each shared expert as one group of all tokens. A token's output reads every
    column of its rows of H and O, so one row per row tile covers every (row tile, column tile)
    pair of both GEMMs, including each group's ragged last tile and the down GEMM's tail-split
    tiles. Per row tile: its first and last rows and ``per_tile - 2`` random ones.
    """
    idx_g = np.asarray(idx_g)
    T, K = idx_g.shape
    g = np.random.default_rng(seed)
    flat = idx_g.reshape(-1)
    groups = [np.flatnonzero(flat == e) // K for e in range(E)]
    groups += [np.arange(T) for _ in range(n_shared)]
    toks = set()
    for rows in groups:
        for j in range(0, rows.size, tile):
            blk = rows[j:j + tile]
            toks.update((int(blk[0]), int(blk[-1])))
            toks.update(int(t) for t in g.choice(blk, min(blk.size, max(0, per_tile - 2)), replace=False))
    return np.array(sorted(toks), dtype=np.int64)


def normalized_max_error(y_gpu: np.ndarray, y_ref: np.ndarray) -> float:
    return float(np.abs(y_gpu - y_ref).max() / max(np.abs(y_ref).max(), 1e-30))


def y_to_f64(y: torch.Tensor) -> np.ndarray:
    return y.float().cpu().numpy().astype(np.float64)
