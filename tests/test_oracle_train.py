"""Pins of the Stage-1 training oracle (CPU only), each independent of its own formulas.

* gradients: central finite differences of the loss L = sum_t <dy_t, y_t> of Eq. 1, with the
  gates computed from p * m (Eq. 2) for a real-valued m and the active sets held fixed, against
  the analytic mask, router-weight and router-input gradients;
* Eq. 3: the matrix diag(pi) - pi pi^T is the finite-difference Jacobian of softmax(m~);
* closed forms: with renormalised gates the router gradient on the active set is
  g_k (dg_k - sum_i g_i dg_i) and zero elsewhere; masked experts get no gradient;
* the sampler: exactly E' distinct experts, E' = E takes all, a dominant logit is always drawn,
  and the empirical inclusion frequencies over many uniform draws match the exact inclusion
  probabilities of sequential sampling without replacement (enumerated over all draw orders);
* accumulation over steps is the sum of the per-step gradients;
* the expert-side backward: central finite differences of the Eq. 1 loss (through the oracle's
  own forward, oracle.ffn.moe_layer) for weight entries of routed and shared experts and for
  input entries; SiLU' against finite differences of SiLU; K = E with all gates equal to 1
  and one expert reduces to a dense SwiGLU MLP whose gradient torch's autograd gives.
"""

import itertools

import numpy as np
import pytest

from oracle import routing as R
from oracle import train as TR


def _problem(T=6, d=5, E=6, K=2, seed=0, gate_mode=R.GATE_RENORM):
    g = np.random.default_rng(seed)
    x = g.standard_normal((T, d))
    w = 0.7 * g.standard_normal((E, d))
    mask = np.zeros(E, np.uint8)
    mask[[0, 2, 3, 5]] = 1
    z = R.router_logits(x, w)
    idx, _, _ = R.route_logits(z, K, R.HARD_MASK, gate_mode, mask=mask)
    dy = g.standard_normal((T, d))
    eo = g.standard_normal((T, K, d))   # expert outputs F_i(x_t), held fixed
    return x, w, mask, idx, dy, eo


def _loss(x, w, m_real, idx, dy, eo, gate_mode):
    """L = sum_t <dy_t, sum_k g_{t,k} F_k>, gates from p * m with the sets idx held fixed."""
    p = R.softmax(x @ w.T)
    L = 0.0
    for t in range(x.shape[0]):
        A = idx[t]
        q = p[t, A] * m_real[A]
        gt = q if gate_mode == R.GATE_P else q / q.sum()
        L += float(dy[t] @ (gt[:, None] * eo[t]).sum(0))
    return L


@pytest.mark.parametrize("gate_mode", [R.GATE_P, R.GATE_RENORM])
def test_gradients_match_finite_differences(gate_mode):
    x, w, mask, idx, dy, eo = _problem(gate_mode=gate_mode)
    out = TR.stage1_backward(x, w, mask, np.zeros(6), idx, dy, eo, gate_mode)
    h = 1e-6
    m0 = mask.astype(np.float64)
    for k in range(6):
        mp, mm = m0.copy(), m0.copy()
        mp[k] += h
        mm[k] -= h
        fd = (_loss(x, w, mp, idx, dy, eo, gate_mode) - _loss(x, w, mm, idx, dy, eo, gate_mode)) / (2 * h)
        assert abs(fd - out["d_mask"][k]) < 1e-6 * max(1.0, abs(fd)), (k, fd, out["d_mask"][k])
    for (e, c) in itertools.product(range(6), range(5)):
        wp, wm = w.copy(), w.copy()
        wp[e, c] += h
        wm[e, c] -= h
        fd = (_loss(x, wp, m0, idx, dy, eo, gate_mode) - _loss(x, wm, m0, idx, dy, eo, gate_mode)) / (2 * h)
        assert abs(fd - out["d_w_router"][e, c]) < 1e-6 * max(1.0, abs(fd))
    for (t, c) in itertools.product(range(6), range(5)):
        xp, xm = x.copy(), x.copy()
        xp[t, c] += h
        xm[t, c] -= h
        fd = (_loss(xp, w, m0, idx, dy, eo, gate_mode) - _loss(xm, w, m0, idx, dy, eo, gate_mode)) / (2 * h)
        assert abs(fd - out["d_x_router"][t, c]) < 1e-6 * max(1.0, abs(fd))


def test_masked_and_unselected_experts_get_no_mask_gradient():
    x, w, mask, idx, dy, eo = _problem(T=8, seed=3)
    out = TR.stage1_backward(x, w, mask, np.zeros(6), idx, dy, eo, R.GATE_RENORM)
    used = np.zeros(6, bool)
    used[np.unique(idx)] = True
    assert np.all(out["d_mask"][~used] == 0.0)
    assert np.all(mask[used] == 1)


def test_renormalised_router_gradient_closed_form():
    x, w, mask, idx, dy, eo = _problem(T=7, seed=5)
    out = TR.stage1_backward(x, w, mask, np.zeros(6), idx, dy, eo, R.GATE_RENORM)
    z = x @ w.T
    for t in range(7):
        A = idx[t]
        ga = np.exp(z[t, A] - z[t, A].max())
        ga /= ga.sum()
        dg = out["dg"][t]
        want = np.zeros(6)
        want[A] = ga * (dg - ga @ dg)
        np.testing.assert_allclose(out["dz"][t], want, atol=1e-12)


def test_ste_matrix_is_the_softmax_jacobian():
    g = np.random.default_rng(1)
    ml = g.standard_normal(7)
    dm = g.standard_normal(7)
    h = 1e-6
    J = np.zeros((7, 7))
    for j in range(7):
        a, b = ml.copy(), ml.copy()
        a[j] += h
        b[j] -= h
        J[:, j] = (TR.mask_distribution(a) - TR.mask_distribution(b)) / (2 * h)
    np.testing.assert_allclose(TR.ste_mask_logits_grad(dm, ml), J.T @ dm, atol=1e-8)
    # equal mask logits (the initialisation): pi uniform, the gradient is dm minus its mean over E
    np.testing.assert_allclose(TR.ste_mask_logits_grad(dm, np.zeros(7)), (dm - dm.mean()) / 7, atol=1e-15)


def test_accumulation_over_steps_is_the_sum():
    ml = np.array([0.3, -0.2, 0.0, 0.5, 0.1, -0.4])
    acc = np.zeros(6)
    parts = []
    for s in range(5):
        x, w, mask, idx, dy, eo = _problem(seed=10 + s)
        d = TR.stage1_backward(x, w, mask, ml, idx, dy, eo, R.GATE_P)["d_mask_logits"]
        acc += d
        parts.append(d)
    np.testing.assert_allclose(acc, np.sum(parts, axis=0), atol=1e-15)


def test_sampler_properties():
    g = np.random.default_rng(2)
    ml = g.standard_normal(8)
    for e_keep in range(1, 9):
        m = TR.sample_mask(ml, g.random(e_keep), e_keep)
        assert m.sum() == e_keep and set(np.unique(m)) <= {0, 1}
    assert TR.sample_mask(ml, g.random(8), 8).sum() == 8
    dom = np.zeros(8)
    dom[5] = 40.0
    for _ in range(20):
        assert TR.sample_mask(dom, g.random(3), 3)[5] == 1
    # a first uniform of 0 takes the first expert; a first uniform just below 1 the last
    assert TR.sample_mask(np.zeros(8), [0.0], 1)[0] == 1
    assert TR.sample_mask(np.zeros(8), [1.0 - 1e-12], 1)[7] == 1
    with pytest.raises(ValueError):
        TR.sample_mask(ml, [0.5], 0)


@pytest.mark.parametrize("E,e_keep", [(5, 2), (5, 3), (6, 4)])
def test_sampler_inclusion_frequencies(E, e_keep):
    ml = np.linspace(-1.2, 1.0, E)
    exact = TR.inclusion_probabilities(ml, e_keep)
    assert abs(exact.sum() - e_keep) < 1e-12
    g = np.random.default_rng(7)
    n = 40000
    counts = np.zeros(E)
    for _ in range(n):
        counts += TR.sample_mask(ml, g.random(e_keep), e_keep)
    freq = counts / n
    sigma = np.sqrt(exact * (1 - exact) / n)
    assert np.all(np.abs(freq - exact) < 5 * sigma + 1e-12), (freq, exact)


def test_uniform_logits_include_each_expert_with_probability_ratio():
    exact = TR.inclusion_probabilities(np.zeros(6), 4)
    np.testing.assert_allclose(exact, 4 / 6, atol=1e-12)


def _moe_problem(seed=0, T=7, d=6, F=5, E=4, K=2, S=1):
    g = np.random.default_rng(seed)
    x = g.standard_normal((T, d))
    wgu = 0.5 * g.standard_normal((E, 2 * F, d))
    wd = 0.5 * g.standard_normal((E, d, F))
    sgu = 0.5 * g.standard_normal((S, 2 * F, d)) if S else None
    sd = 0.5 * g.standard_normal((S, d, F)) if S else None
    idx = np.stack([g.choice(E, K, replace=False) for _ in range(T)])
    gate = g.random((T, K))
    dy = g.standard_normal((T, d))
    return x, wgu, wd, sgu, sd, idx, gate, dy


def test_silu_grad_matches_finite_differences():
    from oracle import ffn as O
    a = np.linspace(-6, 6, 41)
    h = 1e-6
    np.testing.assert_allclose(TR.silu_grad(a), (O.silu(a + h) - O.silu(a - h)) / (2 * h), atol=1e-9)


def test_moe_backward_matches_finite_differences():
    from oracle import ffn as O
    x, wgu, wd, sgu, sd, idx, gate, dy = _moe_problem()
    out = TR.moe_layer_backward(x, idx, gate, dy, wgu, wd, sgu, sd)
    def loss(x, wgu, wd, sgu, sd):
        return float(np.sum(dy * O.moe_layer(x, idx, gate, wgu, wd, sgu, sd)))
    h = 1e-6
    g = np.random.default_rng(1)
    checks = [("x", x, out["dx"]), ("wgu", wgu, out["d_w_gate_up"]), ("wd", wd, out["d_w_down"]),
              ("sgu", sgu, out["d_ws_gate_up"]), ("sd", sd, out["d_ws_down"])]
    for name, arr, grad in checks:
        for _ in range(12):
            pos = tuple(g.integers(0, n) for n in arr.shape)
            args = dict(x=x, wgu=wgu, wd=wd, sgu=sgu, sd=sd)
            plus, minus = arr.copy(), arr.copy()
            plus[pos] += h
            minus[pos] -= h
            fp = loss(**{**args, name: plus})
            fm = loss(**{**args, name: minus})
            fd = (fp - fm) / (2 * h)
            assert abs(fd - grad[pos]) < 1e-6 * max(1.0, abs(fd)), (name, pos, fd, grad[pos])


def test_moe_backward_unselected_expert_gets_zero():
    x, wgu, wd, sgu, sd, idx, gate, dy = _moe_problem(seed=2, E=5, S=0)
    idx[idx == 4] = 0           # expert 4 never chosen
    idx[:, 1] = np.where(idx[:, 0] == idx[:, 1], (idx[:, 0] + 1) % 4, idx[:, 1])
    out = TR.moe_layer_backward(x, idx, gate, dy, wgu, wd)
    assert np.all(out["d_w_gate_up"][4] == 0) and np.all(out["d_w_down"][4] == 0)


def test_dense_mlp_reduction_against_autograd():
    import torch
    x, wgu, wd, _, _, _, _, dy = _moe_problem(seed=3, E=1, K=1, S=0)
    T = x.shape[0]
    out = TR.moe_layer_backward(x, np.zeros((T, 1), int), np.ones((T, 1)), dy, wgu, wd)
    xt = torch.tensor(x, requires_grad=True)
    gu = torch.tensor(wgu[0], requires_grad=True)
    dn = torch.tensor(wd[0], requires_grad=True)
    F = wd.shape[2]
    y = (torch.nn.functional.silu(xt @ gu[:F].T) * (xt @ gu[F:].T)) @ dn.T
    y.backward(torch.tensor(dy))
    np.testing.assert_allclose(out["dx"], xt.grad.numpy(), atol=1e-12)
    np.testing.assert_allclose(out["d_w_gate_up"][0], gu.grad.numpy(), atol=1e-12)
    np.testing.assert_allclose(out["d_w_down"][0], dn.grad.numpy(), atol=1e-12)
