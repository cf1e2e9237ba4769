"""Pins of the FFN / combine oracle against things other than itself (CPU only).

* the expert FFN against torch's own SiLU and linear layers in float64 (a
  library statement of the SwiGLU MLP, non-square shapes so a transposed
  operand cannot pass);
* the gather formulation of the layer (each expert on the tokens that chose
  it) against a dense formulation written here (every expert on every token,
  then a masked, gate-weighted sum);
* K = E with g = p reduces to the p-weighted sum over all experts;
* shared experts add with weight 1 and do not depend on routing.
"""

import numpy as np
import pytest
import torch
import torch.nn.functional as TF

from oracle import ffn as O
from oracle import routing as R


def _weights(g, E, F, d, scale=1.0):
    wgu = g.normal(0, scale / np.sqrt(d), size=(E, 2 * F, d))
    wdn = g.normal(0, scale / np.sqrt(F), size=(E, d, F))
    return wgu, wdn


def test_expert_ffn_matches_torch_swiglu():
    g = np.random.default_rng(0)
    d, F, n = 24, 40, 13
    x = g.normal(size=(n, d))
    wgu, wdn = _weights(g, 1, F, d, 3.0)
    ours = O.expert_ffn(x, wgu[0], wdn[0])
    xt = torch.from_numpy(x)
    ref = TF.linear(TF.silu(TF.linear(xt, torch.from_numpy(wgu[0, :F]))) *
                    TF.linear(xt, torch.from_numpy(wgu[0, F:])), torch.from_numpy(wdn[0]))
    np.testing.assert_allclose(ours, ref.numpy(), rtol=1e-12, atol=1e-12)


def test_silu_against_torch():
    u = np.linspace(-30, 30, 1001)
    np.testing.assert_allclose(O.silu(u), TF.silu(torch.from_numpy(u)).numpy(), rtol=1e-14, atol=1e-300)


@pytest.mark.parametrize("gate_mode", [R.GATE_P, R.GATE_RENORM])
@pytest.mark.parametrize("n_shared", [0, 2])
def test_gather_equals_dense_formulation(gate_mode, n_shared):
    g = np.random.default_rng(10 + gate_mode + n_shared)
    T, d, F, E, K = 37, 16, 24, 6, 2
    x = g.normal(size=(T, d))
    wr = g.normal(0, 0.5, size=(E, d))
    wgu, wdn = _weights(g, E, F, d)
    sgu, sdn = _weights(g, n_shared, F, d)
    idx, gate, _ = R.route(x, wr, K, R.PLAIN, gate_mode)
    y = O.moe_layer(x, idx, gate, wgu, wdn, sgu if n_shared else None, sdn if n_shared else None)
    # dense: every expert on every token, then select with a one-hot gate matrix
    Gm = np.zeros((T, E))
    for t in range(T):
        for k in range(K):
            Gm[t, idx[t, k]] += gate[t, k]
    dense = np.stack([O.expert_ffn(x, wgu[e], wdn[e]) for e in range(E)], axis=1)   # [T,E,d]
    ref = np.einsum("te,ted->td", Gm, dense)
    for s in range(n_shared):
        ref += O.expert_ffn(x, sgu[s], sdn[s])
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


def test_k_equals_e_reduces_to_probability_weighted_sum():
    g = np.random.default_rng(4)
    T, d, F, E = 9, 12, 20, 5
    x = g.normal(size=(T, d))
    wr = g.normal(size=(E, d))
    wgu, wdn = _weights(g, E, F, d)
    idx, gate, _ = R.route(x, wr, E, R.PLAIN, R.GATE_P)
    y = O.moe_layer(x, idx, gate, wgu, wdn)
    p = torch.softmax(torch.from_numpy(x @ wr.T), dim=1).numpy()
    ref = sum(p[:, e:e + 1] * O.expert_ffn(x, wgu[e], wdn[e]) for e in range(E))
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)


def test_shared_experts_add_with_unit_weight():
    g = np.random.default_rng(8)
    T, d, F, E, K = 11, 8, 10, 4, 2
    x = g.normal(size=(T, d))
    wgu, wdn = _weights(g, E, F, d)
    sgu, sdn = _weights(g, 1, F, d)
    idx = np.tile(np.array([[0, 1]]), (T, 1))
    zero_gate = np.zeros((T, K))
    y = O.moe_layer(x, idx, zero_gate, wgu, wdn, sgu, sdn)
    xt = torch.from_numpy(x)
    ref = TF.linear(TF.silu(TF.linear(xt, torch.from_numpy(sgu[0, :F]))) *
                    TF.linear(xt, torch.from_numpy(sgu[0, F:])), torch.from_numpy(sdn[0]))
    np.testing.assert_allclose(y, ref.numpy(), rtol=1e-12, atol=1e-12)


def test_moe_token_equals_batched_layer():
    g = np.random.default_rng(21)
    T, d, F, E, K = 7, 8, 12, 4, 2
    x = g.normal(size=(T, d))
    wgu, wdn = _weights(g, E, F, d)
    idx = np.array([[0, 1], [2, 3], [1, 3], [0, 2], [3, 0], [2, 1], [1, 0]])
    gate = g.random((T, K))
    y = O.moe_layer(x, idx, gate, wgu, wdn)
    for t in range(T):
        np.testing.assert_allclose(O.moe_token(x[t], idx[t], gate[t], wgu, wdn), y[t], rtol=1e-13)
