"""Pins of the LoRA expert oracle (CPU only), independent of its own formula:

* B = 0 (the adapters' initial state) reproduces the base layer exactly;
* an adapted projection equals the plain projection with the merged weight W + (alpha/r) B A,
  so the adapted layer equals oracle.ffn.moe_layer run with merged weights (also with shared
  experts);
* the adapter term is linear in B and scales with alpha / r.
"""

import numpy as np

from oracle import ffn as O


def _problem(seed=0, T=9, d=12, F=10, E=4, K=2, S=1, r=3):
    g = np.random.default_rng(seed)
    x = g.standard_normal((T, d))
    wgu = g.standard_normal((E, 2 * F, d)) / np.sqrt(d)
    wd = g.standard_normal((E, d, F)) / np.sqrt(F)
    sgu = g.standard_normal((S, 2 * F, d)) / np.sqrt(d)
    sd = g.standard_normal((S, d, F)) / np.sqrt(F)
    lora = dict(rank=r, alpha=2.0 * r,
                a_gate_up=g.standard_normal((E, 2 * r, d)), b_gate_up=g.standard_normal((E, 2 * F, r)),
                a_down=g.standard_normal((E, r, F)), b_down=g.standard_normal((E, d, r)),
                as_gate_up=g.standard_normal((S, 2 * r, d)), bs_gate_up=g.standard_normal((S, 2 * F, r)),
                as_down=g.standard_normal((S, r, F)), bs_down=g.standard_normal((S, d, r)))
    idx = np.stack([g.choice(E, K, replace=False) for _ in range(T)])
    gate = g.random((T, K))
    return x, wgu, wd, sgu, sd, lora, idx, gate


def _merge(w_gate_up, w_down, a_gu, b_gu, a_d, b_d, scale, r, F):
    m_gu = w_gate_up.copy()
    m_gu[:F] += scale * b_gu[:F] @ a_gu[:r]
    m_gu[F:] += scale * b_gu[F:] @ a_gu[r:]
    return m_gu, w_down + scale * b_d @ a_d


def test_zero_b_reproduces_the_base_layer():
    x, wgu, wd, sgu, sd, lora, idx, gate = _problem()
    for k in ("b_gate_up", "b_down", "bs_gate_up", "bs_down"):
        lora[k] = np.zeros_like(lora[k])
    np.testing.assert_array_equal(O.lora_moe_layer(x, idx, gate, wgu, wd, lora, sgu, sd),
                                  O.moe_layer(x, idx, gate, wgu, wd, sgu, sd))


def test_adapters_equal_merged_weights():
    x, wgu, wd, sgu, sd, lora, idx, gate = _problem(seed=1)
    r, F = lora["rank"], wd.shape[2]
    scale = lora["alpha"] / r
    mgu, md = wgu.copy(), wd.copy()
    for e in range(wgu.shape[0]):
        mgu[e], md[e] = _merge(wgu[e], wd[e], lora["a_gate_up"][e], lora["b_gate_up"][e], lora["a_down"][e],
                               lora["b_down"][e], scale, r, F)
    smgu, smd = sgu.copy(), sd.copy()
    smgu[0], smd[0] = _merge(sgu[0], sd[0], lora["as_gate_up"][0], lora["bs_gate_up"][0], lora["as_down"][0],
                             lora["bs_down"][0], scale, r, F)
    np.testing.assert_allclose(O.lora_moe_layer(x, idx, gate, wgu, wd, lora, sgu, sd),
                               O.moe_layer(x, idx, gate, mgu, md, smgu, smd), atol=1e-10)


def test_adapter_term_linear_in_b_and_scaled_by_alpha_over_rank():
    g = np.random.default_rng(2)
    x, w = g.standard_normal((5, 7)), g.standard_normal((6, 7))
    a, b = g.standard_normal((3, 7)), g.standard_normal((6, 3))
    base = x @ w.T
    t1 = O.lora_linear(x, w, a, b, 1.0) - base
    np.testing.assert_allclose(O.lora_linear(x, w, a, 2.5 * b, 1.0) - base, 2.5 * t1, atol=1e-12)
    np.testing.assert_allclose(O.lora_linear(x, w, a, b, 16 / 8) - base, 2.0 * t1, atol=1e-12)
