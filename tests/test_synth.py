"""Input generator checks (CPU only): bf16 rounding, determinism, shapes, distributions."""

import numpy as np
import torch

from paper_2609_34077_amd import synth


def test_bf16_rounding_matches_torch():
    g = np.random.default_rng(0)
    a = np.concatenate([g.normal(0, 1, 100000), g.normal(0, 1e-3, 1000), g.normal(0, 1e4, 1000),
                        np.array([0.0, -0.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 65504.0])]).astype(np.float32)
    ours = synth.bf16_bits(a)
    ref = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)
    back = synth.bf16_to_f32(ours)
    np.testing.assert_array_equal(back, torch.from_numpy(ours.view(np.int16)).view(torch.bfloat16).float().numpy())


def test_layer_inputs_deterministic_and_shaped():
    cfg = synth.tiny_config()
    a = synth.make_layer(cfg, threads=1)
    b = synth.make_layer(cfg, threads=4)
    for k in a:
        np.testing.assert_array_equal(a[k], b[k])
    assert a["x"].shape == (64, 256) and a["x"].dtype == np.float32
    assert a["w_router"].shape == (8, 256)
    assert a["w_gate_up"].shape == (8, 1024, 256)
    assert a["w_down"].shape == (8, 256, 512)
    assert a["mask"].tolist() == [1, 0, 1, 0, 0, 1, 0, 1]
    assert abs(a["w_router"].std() - 0.02) < 0.002
    assert abs(a["w_gate_up"].std() - 1 / 16) < 0.002
    assert abs(a["w_down"].std() - 1 / np.sqrt(512)) < 0.002
    assert (a["prior"] > 0).all() and abs(a["prior"].sum() - 1) < 1e-6


def test_deepseek_shapes_small():
    cfg = synth.deepseek_config().with_(T=8, d=64, F=32)
    a = synth.make_layer(cfg)
    assert a["w_gate_up"].dtype == np.uint16
    assert a["ws_gate_up"].shape == (2, 64, 64)
    assert a["ws_down"].shape == (2, 64, 32)
    assert len(cfg.mask_set) == 12 and int(a["mask"].sum()) == 12


def test_trace_inputs_ar1_statistics():
    cfg = synth.TraceConfig(L=3, S=4, N=200, d=256)
    a = synth.make_trace_inputs(cfg)
    x = synth.bf16_to_f32(a["x"]).astype(np.float64).reshape(cfg.S, cfg.N, cfg.d)
    assert abs(x.var() - 1.0) < 0.05
    lag1 = (x[:, 1:] * x[:, :-1]).mean() / x.var()
    assert abs(lag1 - cfg.rho) < 0.02
    assert a["w_router"].shape == (3, 8, 256)
    assert a["prior"].shape == (3, 8)
    for l in range(3):
        s = a["sets"][l]
        assert len(set(s.tolist())) == 4
        assert (a["prior"][l][s] > a["prior"][l].max() - 1e-7).all()


def test_random_trace_distinct_per_step():
    tr = synth.random_trace(2, 3, 50, 3, 8, seed=1, locality=0.5)
    for row in tr.reshape(-1, 3):
        assert len(set(row.tolist())) == 3
        assert ((row >= 0) & (row < 8)).all()
