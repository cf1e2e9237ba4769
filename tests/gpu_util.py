"""Helpers of the GPU parity tests: device upload of synthetic inputs and the comparison
rules against the oracle.

Routing parity rule: where the oracle's margin (gap between the K-th and (K+1)-th
log-domain keys) exceeds 1e-3 logit units the selected expert sets must be identical;
elsewhere several answers are correct and the GPU's set must be a valid Top-K within
1e-3 of the K-th key. Gates are compared per selected expert. Output parity:
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
    for t in range(T):
        if margin_o[t] > MARGIN_TOL:
            if set(idx_g[t].tolist()) != set(idx_o[t].tolist()):
                raise AssertionError(f"token {t}: gpu {idx_g[t]} oracle {idx_o[t]} margin {margin_o[t]}")
            go = dict(zip(idx_o[t].tolist(), gate_o[t].tolist()))
            for j, e in enumerate(idx_g[t].tolist()):
                assert abs(gate_g[t, j] - go[e]) <= gate_rtol * max(abs(go[e]), 1e-30) + 1e-7, (t, e)
        else:
            near += 1
            assert R.valid_selection(z[t], idx_g[t], K, mode, mask, prior, MARGIN_TOL), (t, idx_g[t])
    if margin_g is not None:
        mg = np.asarray(margin_g, dtype=np.float64)
        fin = np.isfinite(margin_o)
        assert (np.isinf(mg) == ~fin).all()
        assert np.abs(mg[fin] - margin_o[fin]).max(initial=0.0) <= margin_atol
    return near


def normalized_max_error(y_gpu: np.ndarray, y_ref: np.ndarray) -> float:
    return float(np.abs(y_gpu - y_ref).max() / max(np.abs(y_ref).max(), 1e-30))


def y_to_f64(y: torch.Tensor) -> np.ndarray:
    return y.float().cpu().numpy().astype(np.float64)
