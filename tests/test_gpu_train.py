"""GPU parity of the Stage 1 training entry points (Section 3.2, Eq. 2 and Eq. 3).

* maskmoe_stage1_backward against the oracle on the same inputs: seeded x, router, dy and
  expert outputs, with the routing sets and logits taken from the oracle's own routing, at small
  sizes (ragged, both gate rules, bf16 and f32) and at the full Mixtral-shaped fine-tuning size
  (8192 tokens, d = 4096) and DeepSeek-shaped size. Bounds: fp32 accumulation, so each output's
  error is bounded by 1e-4 (1e-5 for single dot products) times the sum of the absolute values
  of the terms it adds up.
* maskmoe_layer_forward_train: the logits and per-slot expert outputs against the oracle, y
  identical to maskmoe_layer_forward.
* the whole step end to end (GPU forward, then GPU backward) against the oracle's forward and
  backward, on a case without near-ties (identical routing sets).
"""

import numpy as np
import pytest
import torch

import gpu_util as U
from oracle import ffn as O
from oracle import routing as R
from oracle import train as TR
from paper_2609_34077_amd import _lib as L
from paper_2609_34077_amd import synth

pytestmark = pytest.mark.gpu


def _case(T, d, E, K, gate_mode, dtype, keep, seed):
    g = np.random.default_rng(seed)
    x = g.standard_normal((T, d)).astype(np.float32)
    w = (0.02 * g.standard_normal((E, d))).astype(np.float32)
    dy = g.standard_normal((T, d)).astype(np.float32)
    eo = g.standard_normal((T, K, d)).astype(np.float32)
    ml = (0.5 * g.standard_normal(E)).astype(np.float32)
    acc0 = g.standard_normal(E).astype(np.float32)
    if dtype == "bf16":
        x, w, dy = synth.bf16_bits(x), synth.bf16_bits(w), synth.bf16_bits(dy)
    mask = synth.binary_mask(E, keep)
    return dict(x=x, w=w, dy=dy, eo=eo, ml=ml, acc0=acc0, mask=mask)


def _bound_ok(got, want, scale, rel, what):
    err = np.abs(np.asarray(got, np.float64) - want)
    lim = rel * scale + 1e-12
    bad = err > lim
    assert not bad.any(), f"{what}: {bad.sum()} of {bad.size} beyond bound, worst {(err / lim).max():.3g}x"


def _check_backward(c, K, gate_mode, dtype):
    xf, wf, dyf = U.f64(c["x"], dtype), U.f64(c["w"], dtype), U.f64(c["dy"], dtype)
    z = R.router_logits(xf, wf)
    idx, _, _ = R.route_logits(z, K, R.HARD_MASK, gate_mode, mask=c["mask"])
    ref = TR.stage1_backward(xf, wf, c["mask"], c["ml"].astype(np.float64), idx, dyf, c["eo"], gate_mode)
    acc = torch.from_numpy(c["acc0"].copy()).cuda()
    out = L.maskmoe_stage1_backward(U.dev(c["x"]), U.dev(c["w"]), K, gate_mode, c["mask"],
                                    torch.from_numpy(idx.astype(np.int32)).cuda(),
                                    torch.from_numpy(z.astype(np.float32)).cuda(), U.dev(c["dy"]),
                                    U.dev(c["eo"]), mask_logits=c["ml"], d_mask_logits=acc)
    torch.cuda.synchronize()
    eo = c["eo"].astype(np.float64)
    dg_scale = np.einsum("td,tkd->tk", np.abs(dyf), np.abs(eo))
    _bound_ok(out["d_gate"].cpu().numpy(), ref["dg"], dg_scale, 1e-5, "d_gate")
    term = 2.0 * np.abs(ref["dg"]).sum()          # every per-token mask / logit term is <= 2 |dg|
    _bound_ok(out["d_mask"].cpu().numpy(), ref["d_mask"], term, 1e-4, "d_mask")
    want_acc = c["acc0"].astype(np.float64) + ref["d_mask_logits"]
    _bound_ok(acc.cpu().numpy(), want_acc, 2.0 * term + np.abs(c["acc0"]), 1e-4, "d_mask_logits")
    # dz_t is a difference of terms of size ~|dg_t| (for K = 2 renormalised gates it is
    # g_a g_b (dg_a - dg_b)), so its rounding error scales with s_t = sum_k |dg_{t,k}|, not with
    # |dz_t|; the router gradients inherit that error through dW = dz^T x and dx = dz W.
    s = np.abs(ref["dg"]).sum(1)
    dz_err = np.abs(ref["dz"]) + s[:, None]
    _bound_ok(out["d_w_router"].cpu().numpy(), ref["d_w_router"], dz_err.T @ np.abs(xf) + 1e-30, 1e-4, "d_w_router")
    _bound_ok(out["d_x"].cpu().numpy(), ref["d_x_router"], dz_err @ np.abs(wf) + 1e-30, 1e-4, "d_x")
    return out


BACKWARD_CASES = [
    ("mixtral_shaped_small", 300, 256, 8, 2, R.GATE_RENORM, "bf16", (0, 2, 5, 7)),
    ("deepseek_shaped_small", 200, 512, 64, 6, R.GATE_P, "bf16", tuple(synth.deepseek_mask_set())),
    ("tiny_f32", 64, 256, 8, 2, R.GATE_RENORM, "f32", (0, 2, 5, 7)),
    ("gate_p_f32_ragged", 77, 96, 16, 3, R.GATE_P, "f32", tuple(range(0, 16, 2))),
    ("scalar_load_paths_bf16", 70, 98, 8, 2, R.GATE_RENORM, "bf16", (0, 2, 5, 7)),   # rows not vector aligned
]


@pytest.mark.parametrize("name,T,d,E,K,gate_mode,dtype,keep", BACKWARD_CASES, ids=[c[0] for c in BACKWARD_CASES])
def test_stage1_backward_matches_oracle(name, T, d, E, K, gate_mode, dtype, keep):
    U.say(f"stage1 backward {name} T={T} d={d} E={E} K={K} gate={gate_mode} {dtype}")
    _check_backward(_case(T, d, E, K, gate_mode, dtype, keep, seed=T + E), K, gate_mode, dtype)


def test_stage1_backward_accumulates_and_is_deterministic():
    c = _case(129, 256, 8, 2, R.GATE_RENORM, "bf16", (1, 3, 4, 6), seed=4)
    xf, wf = U.f64(c["x"], "bf16"), U.f64(c["w"], "bf16")
    z = R.router_logits(xf, wf)
    idx, _, _ = R.route_logits(z, 2, R.HARD_MASK, R.GATE_RENORM, mask=c["mask"])
    args = (U.dev(c["x"]), U.dev(c["w"]), 2, R.GATE_RENORM, c["mask"], torch.from_numpy(idx.astype(np.int32)).cuda(),
            torch.from_numpy(z.astype(np.float32)).cuda(), U.dev(c["dy"]), U.dev(c["eo"]))
    acc = torch.zeros(8, dtype=torch.float32, device="cuda")
    a = L.maskmoe_stage1_backward(*args, mask_logits=c["ml"], d_mask_logits=acc)
    once = acc.clone()
    b = L.maskmoe_stage1_backward(*args, mask_logits=c["ml"], d_mask_logits=acc)
    torch.cuda.synchronize()
    for k in ("d_gate", "d_mask", "d_w_router", "d_x"):
        assert torch.equal(a[k], b[k]), k
    assert torch.equal(acc, once + once)


@pytest.mark.parametrize("name,T,d,E,K,gate_mode,keep", [
    ("mixtral_ft_t8192", 8192, 4096, 8, 2, R.GATE_RENORM, (0, 2, 5, 7)),
    ("deepseek_t4096", 4096, 2048, 64, 6, R.GATE_P, tuple(synth.deepseek_mask_set())),
])
def test_stage1_backward_full_size(name, T, d, E, K, gate_mode, keep):
    U.say(f"stage1 backward full size {name}")
    _check_backward(_case(T, d, E, K, gate_mode, "bf16", keep, seed=11), K, gate_mode, "bf16")


def _layer(cfg):
    inp = synth.make_layer(cfg)
    dd = {k: U.dev(inp[k]) for k in ("x", "w_router", "w_gate_up", "w_down")}
    return inp, dd


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_forward_train_outputs(dtype):
    cfg = synth.LayerConfig(f"train_fwd_{dtype}", T=48, d=256, F=512, E=8, K=2, dtype=dtype,
                            route_mode=L.ROUTE_HARD_MASK, mask_set=(0, 2, 5, 7), seed=33)
    U.say(f"forward_train {cfg.name}")
    inp, dd = _layer(cfg)
    y, idx, gate, logits, eo = L.maskmoe_layer_forward_train(dd["x"], dd["w_router"], dd["w_gate_up"], dd["w_down"],
                                                             cfg.K, cfg.route_mode, cfg.gate_mode, mask=inp["mask"])
    y_plain = L.maskmoe_layer_forward(dd["x"], dd["w_router"], dd["w_gate_up"], dd["w_down"], cfg.K,
                                      cfg.route_mode, cfg.gate_mode, mask=inp["mask"])
    torch.cuda.synchronize()
    assert torch.equal(y, y_plain)
    xf = U.f64(inp["x"], dtype)
    z = R.router_logits(xf, U.f64(inp["w_router"], dtype))
    lg = logits.cpu().numpy().astype(np.float64)
    np.testing.assert_allclose(lg, z, atol=1e-5 * np.abs(z).max())
    idx_o, _, margin_o = R.route_logits(z, cfg.K, R.HARD_MASK, cfg.gate_mode, mask=inp["mask"])
    assert (margin_o > U.MARGIN_TOL).all(), "this seed must have no near-ties"
    assert np.array_equal(np.sort(idx.cpu().numpy(), 1), np.sort(idx_o, 1))
    eo_g = eo.cpu().numpy().astype(np.float64)
    wgu, wdn = inp["w_gate_up"], inp["w_down"]
    tol = U.BF16_TOL if dtype == "bf16" else U.F32_TOL
    idx_g = idx.cpu().numpy()
    for e in range(cfg.E):
        sel = np.argwhere(idx_g == e)
        if len(sel) == 0:
            continue
        ref = O.expert_ffn(xf[sel[:, 0]], U.f64(wgu[e], dtype), U.f64(wdn[e], dtype))
        got = eo_g[sel[:, 0], sel[:, 1]]
        assert np.abs(got - ref).max() <= tol * np.abs(ref).max(), e


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_training_step_end_to_end(dtype):
    cfg = synth.LayerConfig(f"train_step_{dtype}", T=48, d=256, F=512, E=8, K=2, dtype=dtype,
                            route_mode=L.ROUTE_HARD_MASK, mask_set=(0, 2, 5, 7), seed=33)
    U.say(f"training step end to end {cfg.name}")
    inp, dd = _layer(cfg)
    g = np.random.default_rng(5)
    dy = g.standard_normal((cfg.T, cfg.d)).astype(np.float32)
    dy = synth.bf16_bits(dy) if dtype == "bf16" else dy
    ml = (0.3 * g.standard_normal(cfg.E)).astype(np.float32)
    y, idx, gate, logits, eo = L.maskmoe_layer_forward_train(dd["x"], dd["w_router"], dd["w_gate_up"], dd["w_down"],
                                                             cfg.K, cfg.route_mode, cfg.gate_mode, mask=inp["mask"])
    acc = torch.zeros(cfg.E, dtype=torch.float32, device="cuda")
    out = L.maskmoe_stage1_backward(dd["x"], dd["w_router"], cfg.K, cfg.gate_mode, inp["mask"], idx, logits,
                                    U.dev(dy), eo, mask_logits=ml, d_mask_logits=acc)
    torch.cuda.synchronize()
    # the oracle's own forward: routing, then every selected expert's output in float64
    xf, wf, dyf = U.f64(inp["x"], dtype), U.f64(inp["w_router"], dtype), U.f64(dy, dtype)
    z = R.router_logits(xf, wf)
    idx_o, _, margin_o = R.route_logits(z, cfg.K, R.HARD_MASK, cfg.gate_mode, mask=inp["mask"])
    assert (margin_o > U.MARGIN_TOL).all()
    assert np.array_equal(idx.cpu().numpy(), idx_o)
    eo_o = np.zeros((cfg.T, cfg.K, cfg.d))
    for t in range(cfg.T):
        for k in range(cfg.K):
            e = idx_o[t, k]
            eo_o[t, k] = O.expert_ffn(xf[t:t + 1], U.f64(inp["w_gate_up"][e], dtype), U.f64(inp["w_down"][e], dtype))[0]
    ref = TR.stage1_backward(xf, wf, inp["mask"], ml.astype(np.float64), idx_o, dyf, eo_o, cfg.gate_mode)
    tol = 2 * U.BF16_TOL if dtype == "bf16" else 1e-4
    for k_out, k_ref in (("d_mask", "d_mask"), ("d_w_router", "d_w_router"), ("d_x", "d_x_router"),
                         ("d_gate", "dg")):
        got = out[k_out].cpu().numpy().astype(np.float64)
        want = ref[k_ref]
        assert np.abs(got - want).max() <= tol * np.abs(want).max(), k_out
    got = acc.cpu().numpy().astype(np.float64)
    assert np.abs(got - ref["d_mask_logits"]).max() <= tol * np.abs(ref["d_mask_logits"]).max()
