"""Oracle: what an offloaded decode step moves and computes (float64 / pure Python).
Test infrastructure only.

Section 1 and Section 3.1: experts live in host memory and a layer keeps B of them on the GPU;
at every decode step each selected expert that is not cached is fetched over PCIe (one transfer
of all its weights), and a full cache evicts one cached expert per fetch under the policy
(Section 4.1: LRU, LFU, FIFO). The step's output is Eq. 1 on the same weights: offloading
changes where the weights are read from, not what the layer computes.

``decode_steps`` runs a batch-1 decode of one layer over a token sequence: routing of each
token (Eq. 1, 2 or 4 per the rule), the cache step of ``oracle.cache`` on its selected set, and
the layer output. The policy rules and their readings are those of ``oracle.cache``.
"""

from __future__ import annotations

from typing import Callable, Optional

import numpy as np

from . import cache as C
from . import ffn as O
from . import routing as R


def expert_bytes(d: int, F: int, elem_bytes: int = 2) -> int:
    """Bytes of one SwiGLU expert (W_gate, W_up [F, d] and W_down [d, F])."""
    return 3 * d * F * elem_bytes


def decode_steps(xs, w_router, w_gate_up, w_down, K: int, route_mode: int, gate_mode: int, B: int,
                 policy: int, mask=None, prior=None, ws_gate_up=None, ws_down=None, state=None, counts=None,
                 widen: Optional[Callable] = None):
    """Decode tokens xs [N, d] one at a time through one layer with a B-expert cache.

    Returns dict(idx [N,K], gate [N,K], margin [N], y [N,d], fetched (per step, the experts
    fetched in insertion order), evicted (per step), cache (per step, the state after it),
    f [N], h [N], final_state, final_counts).
    """
    xs = np.asarray(xs, dtype=np.float64)
    wr = np.asarray(w_router, dtype=np.float64)
    E = wr.shape[0]
    z = R.router_logits(xs, wr)
    idx, gate, margin = R.route_logits(z, K, route_mode, gate_mode, mask=mask, prior=prior)
    traj: list = []
    f, h, final, freq, bad = C.replay_stream(idx.tolist(), E, B, policy, state, counts, trajectory=traj)
    if bad:
        raise ValueError("routing produced an invalid step")
    y = O.moe_layer(xs, idx, gate, w_gate_up, w_down, ws_gate_up, ws_down, widen=widen)
    return dict(idx=idx, gate=gate, margin=margin, y=y, fetched=[t["fetched"] for t in traj],
                evicted=[t["evicted"] for t in traj], cache=[t["cache"] for t in traj], f=np.asarray(f),
                h=np.asarray(h), final_state=final, final_counts=freq)
