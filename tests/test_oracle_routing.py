"""Pins of the routing oracle against things other than itself (CPU only).

* brute force over every K-subset of experts (the Top-K of Eq. 1, Eq. 2 and
  Eq. 4 is the subset whose every key beats every key outside it);
* the closed form of top-2 renormalised gates (a logistic of the logit gap);
* library softmax (scipy) for the gate values;
* invariants the paper states: gates under the hard mask equal the gates of
  p on the active set (Section 3.2, Stage 1); the prior excludes no expert
  and does not change gate values (Section 3.2, Evaluation and inference);
* special cases: an all-ones mask and a uniform prior reduce to plain
  Top-K; a mask with exactly K ones selects the mask set; a very strong
  prior reduces to the hard mask;
* hand-worked examples in ``tests/golden/routing_hand_examples.txt``.
"""

import itertools
import math

import numpy as np
import pytest
from scipy.special import expit, softmax as sp_softmax

from conftest import golden_path
from oracle import routing as R


def _brute_force_set(keys_row, K, eligible):
    """The unique K-subset S of eligible experts with min key(S) > max key(eligible \\ S)."""
    cand = [i for i in range(len(keys_row)) if eligible[i]]
    winners = []
    for S in itertools.combinations(cand, K):
        rest = [i for i in cand if i not in S]
        if not rest or min(keys_row[i] for i in S) > max(keys_row[i] for i in rest):
            winners.append(set(S))
    assert len(winners) == 1
    return winners[0]


@pytest.mark.parametrize("E,K", [(4, 1), (4, 2), (6, 2), (8, 2), (8, 3), (10, 4)])
@pytest.mark.parametrize("mode", [R.PLAIN, R.HARD_MASK, R.SOFT_PRIOR])
def test_topk_matches_brute_force(E, K, mode):
    g = np.random.default_rng(1000 * E + 10 * K + mode)
    T = 40
    z = g.normal(0.0, 1.5, size=(T, E))
    mask = np.zeros(E, np.uint8)
    mask[g.choice(E, size=max(K, E - 2), replace=False)] = 1
    prior = sp_softmax(g.normal(0, 1.0, size=E))
    idx, gate, margin = R.route_logits(z, K, mode, R.GATE_RENORM, mask=mask, prior=prior)
    p = sp_softmax(z, axis=1)
    for t in range(T):
        if mode == R.PLAIN:
            keys, elig = p[t], np.ones(E, bool)
        elif mode == R.HARD_MASK:
            keys, elig = p[t] * mask, mask.astype(bool)
        else:
            keys, elig = p[t] * prior, np.ones(E, bool)
        assert set(idx[t].tolist()) == _brute_force_set(keys, K, elig)
        # listed by decreasing key
        assert all(keys[idx[t][j]] >= keys[idx[t][j + 1]] for j in range(K - 1))


def test_renorm_top2_closed_form():
    g = np.random.default_rng(7)
    z = g.normal(0, 2.0, size=(200, 8))
    idx, gate, _ = R.route_logits(z, 2, R.PLAIN, R.GATE_RENORM)
    za = np.take_along_axis(z, idx, axis=1)
    np.testing.assert_allclose(gate[:, 0], expit(za[:, 0] - za[:, 1]), rtol=1e-13, atol=0)
    np.testing.assert_allclose(gate[:, 1], expit(za[:, 1] - za[:, 0]), rtol=1e-12, atol=0)


@pytest.mark.parametrize("mode", [R.PLAIN, R.HARD_MASK, R.SOFT_PRIOR])
def test_gates_come_from_full_softmax(mode):
    g = np.random.default_rng(11 + mode)
    E, K = 16, 4
    z = g.normal(0, 1.0, size=(64, E))
    mask = np.zeros(E, np.uint8)
    mask[[1, 3, 4, 8, 9, 15]] = 1
    prior = sp_softmax(g.normal(0, 2.0, size=E))
    idx, gp, _ = R.route_logits(z, K, mode, R.GATE_P, mask=mask, prior=prior)
    _, gr, _ = R.route_logits(z, K, mode, R.GATE_RENORM, mask=mask, prior=prior)
    p = sp_softmax(z, axis=1)
    sel = np.take_along_axis(p, idx, axis=1)
    np.testing.assert_allclose(gp, sel, rtol=1e-13)
    np.testing.assert_allclose(gr.sum(axis=1), 1.0, rtol=1e-13)
    np.testing.assert_allclose(gr, sel / sel.sum(axis=1, keepdims=True), rtol=1e-13)
    if mode == R.HARD_MASK:
        # Gates from p*m equal the gates from p on the active set (Stage 1).
        pm = p * mask
        np.testing.assert_allclose(np.take_along_axis(pm, idx, axis=1), gp, rtol=0, atol=0)
        assert mask[idx].all()


def test_all_ones_mask_and_uniform_prior_reduce_to_plain():
    g = np.random.default_rng(3)
    E, K = 8, 2
    z = g.normal(0, 1.3, size=(500, E))
    ip, gp, mp = R.route_logits(z, K, R.PLAIN, R.GATE_RENORM)
    ih, gh, mh = R.route_logits(z, K, R.HARD_MASK, R.GATE_RENORM, mask=np.ones(E, np.uint8))
    iu, gu, mu = R.route_logits(z, K, R.SOFT_PRIOR, R.GATE_RENORM, prior=np.full(E, 1.0 / E))
    assert (ip == ih).all() and (ip == iu).all()
    np.testing.assert_array_equal(gp, gh)
    np.testing.assert_allclose(gp, gu, rtol=1e-15)
    np.testing.assert_array_equal(mp, mh)
    np.testing.assert_allclose(mp, mu, rtol=1e-12)


def test_mask_with_exactly_k_ones_selects_the_mask_set():
    g = np.random.default_rng(5)
    E, K = 64, 6
    keep = sorted(g.choice(E, K, replace=False).tolist())
    mask = np.zeros(E, np.uint8)
    mask[keep] = 1
    z = g.normal(0, 1.0, size=(100, E))
    idx, _, margin = R.route_logits(z, K, R.HARD_MASK, R.GATE_P, mask=mask)
    for t in range(100):
        assert sorted(idx[t].tolist()) == keep
    assert np.isinf(margin).all()


def test_strong_prior_reduces_to_hard_mask():
    g = np.random.default_rng(9)
    E, K = 8, 2
    keep = [0, 2, 5, 7]
    mask = np.zeros(E, np.uint8)
    mask[keep] = 1
    ml = np.zeros(E)
    ml[keep] = 60.0
    prior = sp_softmax(ml)
    z = g.normal(0, 1.3, size=(400, E))
    ih, gh, _ = R.route_logits(z, K, R.HARD_MASK, R.GATE_RENORM, mask=mask)
    iss, gs, _ = R.route_logits(z, K, R.SOFT_PRIOR, R.GATE_RENORM, prior=prior)
    assert (ih == iss).all()
    np.testing.assert_allclose(gh, gs, rtol=1e-15)


def test_prior_excludes_no_expert():
    # An expert outside the favoured set is still selected when its p_i * pi_i
    # ranks among the K largest (Section 3.2, Evaluation and inference).
    E, K = 8, 2
    keep = [1, 2, 3, 4]
    prior = sp_softmax(np.where(np.isin(np.arange(E), keep), 1.0, 0.0))
    z = np.zeros((1, E))
    z[0, 6] = 5.0                        # far above everyone: e^5 > e^1
    idx, _, _ = R.route_logits(z, K, R.SOFT_PRIOR, R.GATE_RENORM, prior=prior)
    assert 6 in idx[0].tolist()
    assert R.route_logits(z, K, R.HARD_MASK, R.GATE_RENORM,
                          mask=np.isin(np.arange(E), keep).astype(np.uint8))[0][0].tolist() != [6]


def test_log_keys_rank_like_literal_products():
    g = np.random.default_rng(17)
    E, K = 8, 2
    z = g.normal(0, 1.3, size=(3000, E))
    prior = sp_softmax(g.normal(0, 1.0, size=E))
    mask = (g.random(E) < 0.6).astype(np.uint8)
    mask[:K] = 1
    for mode in (R.PLAIN, R.HARD_MASK, R.SOFT_PRIOR):
        idx, _, margin = R.route_logits(z, K, mode, R.GATE_P, mask=mask, prior=prior)
        lit = R.literal_keys(sp_softmax(z, axis=1), mode, mask, prior)
        order = np.argsort(-lit, axis=1, kind="stable")[:, :K]
        ok = margin > 1e-9
        assert (np.sort(order[ok], 1) == np.sort(idx[ok], 1)).all()


def test_margin_is_kth_minus_next_log_key():
    z = np.array([[3.0, -1.0, 2.5, 0.25, 2.0]])
    idx, _, margin = R.route_logits(z, 2, R.PLAIN, R.GATE_P)
    assert idx[0].tolist() == [0, 2]
    assert margin[0] == pytest.approx(0.5)
    idx, _, margin = R.route_logits(z, 3, R.PLAIN, R.GATE_P)
    assert margin[0] == pytest.approx(1.75)
    idx, _, margin = R.route_logits(z, 5, R.PLAIN, R.GATE_P)
    assert np.isinf(margin[0])


def test_equal_keys_go_to_lower_index():
    z = np.array([[1.0, 2.0, 2.0, 2.0, 0.0]])
    idx, _, margin = R.route_logits(z, 2, R.PLAIN, R.GATE_P)
    assert idx[0].tolist() == [1, 2]
    assert margin[0] == 0.0


def _read_hand_examples():
    rows = []
    with open(golden_path("routing_hand_examples.txt")) as fh:
        for line in fh:
            if line.startswith("#") or not line.strip():
                continue
            name, z, mode, m, sel, margin, gp, gr = [f.strip() for f in line.split("|")]
            rows.append(dict(name=name, z=np.array([float(v) for v in z.split()]),
                             mode={"plain": R.PLAIN, "hard": R.HARD_MASK, "soft": R.SOFT_PRIOR}[mode],
                             m=None if m == "-" else np.array([float(v) for v in m.split()]),
                             sel=[int(v) for v in sel.split()], margin=float(margin),
                             gp=[float(v) for v in gp.split()], gr=[float(v) for v in gr.split()]))
    return rows


@pytest.mark.parametrize("ex", _read_hand_examples(), ids=lambda e: e["name"])
def test_hand_worked_examples(ex):
    z = ex["z"][None, :]
    mask = prior = None
    if ex["mode"] == R.HARD_MASK:
        mask = ex["m"].astype(np.uint8)
    elif ex["mode"] == R.SOFT_PRIOR:
        w = np.exp(ex["m"])
        prior = w / w.sum()
    idx, gp, margin = R.route_logits(z, 2, ex["mode"], R.GATE_P, mask=mask, prior=prior)
    _, gr, _ = R.route_logits(z, 2, ex["mode"], R.GATE_RENORM, mask=mask, prior=prior)
    assert set(idx[0].tolist()) == set(ex["sel"])
    if math.isinf(ex["margin"]):
        assert np.isinf(margin[0])
    else:
        assert margin[0] == pytest.approx(ex["margin"], abs=1e-12)
    # compare gate values as a set-ordered pair (order inside a tie is not unique)
    order = np.argsort(idx[0])
    exp_order = np.argsort(ex["sel"])
    np.testing.assert_allclose(gp[0][order], np.array(ex["gp"])[exp_order], atol=5e-11)
    np.testing.assert_allclose(gr[0][order], np.array(ex["gr"])[exp_order], atol=5e-11)


def test_valid_selection_accepts_near_ties_only():
    z = np.array([1.0, 0.9995, 0.2, -1.0])
    assert R.valid_selection(z, [0, 1], 2, R.PLAIN)
    assert R.valid_selection(z, [0, 2], 1 + 1, R.PLAIN) is False
    z2 = np.array([1.0, 0.5, 0.4996, -1.0])
    assert R.valid_selection(z2, [0, 2], 2, R.PLAIN)       # 2 is within 1e-3 of the K-th
    assert not R.valid_selection(z2, [0, 3], 2, R.PLAIN)
    assert not R.valid_selection(z2, [0, 0], 2, R.PLAIN)
    assert not R.valid_selection(z2, [0, 1], 2, R.HARD_MASK, mask=np.array([1, 0, 1, 1]))


@pytest.mark.parametrize("mode", [R.HARD_MASK, R.SOFT_PRIOR, R.PLAIN])
def test_route_layers_brute_force_per_layer(mode):
    """route_layers routes the same tokens through L independent routers, each with its own
    mask or prior (Section 3.1: every MoE layer has its own router; Section 3.2: one mask and
    prior per layer). Every (layer, token) is checked by brute force over K-subsets with that
    layer's own logits x W_l^T (written out here as explicit dot products) and its own
    mask / prior, and the gates against scipy's softmax of those logits. The layers' masks,
    priors and routers differ, so applying layer 0's mask or prior to every layer, or
    swapping the layer and token axes, fails."""
    g = np.random.default_rng(4242 + mode)
    Lyr, T, d, E, K = 4, 24, 12, 6, 2
    x = g.normal(0, 1.0, size=(T, d))
    w = g.normal(0, 0.6, size=(Lyr, E, d))
    masks = np.zeros((Lyr, E), np.uint8)
    for l, keep in enumerate([(0, 1, 2), (3, 4, 5), (0, 2, 4), (1, 3, 5)]):
        masks[l, list(keep)] = 1
    priors = np.stack([sp_softmax(np.where(masks[l] == 1, 3.0, 0.0)) for l in range(Lyr)])
    idx, gate, margin = R.route_layers(x, w, K, mode, R.GATE_RENORM,
                                       masks=masks if mode == R.HARD_MASK else None,
                                       priors=priors if mode == R.SOFT_PRIOR else None)
    assert idx.shape == (Lyr, T, K) and gate.shape == (Lyr, T, K) and margin.shape == (Lyr, T)
    sets_differ = 0
    for l in range(Lyr):
        for t in range(T):
            z = np.array([sum(x[t, j] * w[l, e, j] for j in range(d)) for e in range(E)])
            p = sp_softmax(z)
            if mode == R.PLAIN:
                keys, elig = p, np.ones(E, bool)
            elif mode == R.HARD_MASK:
                keys, elig = p * masks[l], masks[l].astype(bool)
            else:
                keys, elig = p * priors[l], np.ones(E, bool)
            want = _brute_force_set(keys, K, elig)
            assert set(idx[l, t].tolist()) == want, (l, t)
            sel = [int(e) for e in idx[l, t]]
            np.testing.assert_allclose(gate[l, t], p[sel] / p[sel].sum(), rtol=1e-12)
            if mode == R.HARD_MASK:
                assert all(masks[l, e] for e in sel)
            if set(idx[l, t].tolist()) != set(idx[0, t].tolist()):
                sets_differ += 1
    # the layers really route differently, so a layer mix-up cannot pass unnoticed
    assert sets_differ >= T
    # layer by layer, the result is the single-router routing of that layer
    for l in range(Lyr):
        i1, g1, m1 = R.route(x, w[l], K, mode, R.GATE_RENORM,
                             mask=masks[l] if mode == R.HARD_MASK else None,
                             prior=priors[l] if mode == R.SOFT_PRIOR else None)
        assert np.array_equal(i1, idx[l]) and np.array_equal(g1, gate[l]) and np.array_equal(m1, margin[l])
