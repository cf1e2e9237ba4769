"""GPU parity of maskmoe_layer_forward_lora (Stage 2: every routed and shared expert carries
low-rank adapters on its gate, up and down projections) against the oracle's lora_moe_layer.

Both sides route on their own. Near-tie tokens (oracle margin <= 1e-3) are evaluated by the
oracle on the GPU's validated set with gates from its own p (gpu_util.effective_routing), so
no token is left out. At the full shape the compared tokens cover every 256-row tile of every
expert group. Bound: max-normalised error
<= 1e-2 (bf16 storage; the GPU rounds A x, A h and (alpha / r) B to bf16, the oracle rounds
nothing).
"""

import functools

import numpy as np
import pytest
import torch

import gpu_util as U
from oracle import ffn as O
from oracle import routing as R
from paper_2609_34077_amd import _lib as L
from paper_2609_34077_amd import synth

pytestmark = pytest.mark.gpu


def _mp(cfg, inp):
    if cfg.route_mode == L.ROUTE_HARD_MASK:
        return dict(mask=inp["mask"])
    if cfg.route_mode == L.ROUTE_SOFT_PRIOR:
        return dict(prior=inp["prior"])
    return {}


def _upload_lora(lora, n_shared):
    out = dict(rank=lora["rank"], alpha=lora["alpha"])
    for k in L.LORA_KEYS:
        if n_shared or not k.startswith(("as_", "bs_")):
            out[k] = U.dev(lora[k])
    return out


def _run(cfg, inp, lora_np, workspace=None):
    dd = {k: U.dev(inp[k]) for k in ("x", "w_router", "w_gate_up", "w_down")}
    sgu = U.dev(inp["ws_gate_up"]) if cfg.n_shared else None
    sdn = U.dev(inp["ws_down"]) if cfg.n_shared else None
    idx = torch.empty((cfg.T, cfg.K), dtype=torch.int32, device="cuda")
    gate = torch.empty((cfg.T, cfg.K), dtype=torch.float32, device="cuda")
    y = L.maskmoe_layer_forward_lora(dd["x"], dd["w_router"], dd["w_gate_up"], dd["w_down"], cfg.K, cfg.route_mode,
                                     cfg.gate_mode, _upload_lora(lora_np, cfg.n_shared), ws_gate_up=sgu, ws_down=sdn,
                                     topk_idx=idx, topk_gate=gate, workspace=workspace, **_mp(cfg, inp))
    torch.cuda.synchronize()
    return y, idx, gate


def check_lora(cfg, rank=8, alpha=16.0, sample=False, seed=0):
    U.say(f"lora layer {cfg.name} T={cfg.T} d={cfg.d} F={cfg.F} E={cfg.E} K={cfg.K} shared={cfg.n_shared} "
          f"rank={rank} alpha={alpha}")
    inp = synth.make_layer(cfg)
    lora = synth.make_lora(cfg, rank, alpha)
    y, idx, gate = _run(cfg, inp, lora)
    xf = U.f64(inp["x"], "bf16")
    mp = _mp(cfg, inp)
    z = R.router_logits(xf, U.f64(inp["w_router"], "bf16"))
    ig = idx.cpu().numpy()
    U.check_routing(z, ig, gate.cpu().numpy(), None, cfg.K, cfg.route_mode, cfg.gate_mode, mp.get("mask"),
                    mp.get("prior"))
    io, go, near = U.effective_routing(z, ig, cfg.K, cfg.route_mode, cfg.gate_mode, mp.get("mask"),
                                       mp.get("prior"))
    toks = np.arange(cfg.T)
    if sample:
        toks = U.tile_sample_tokens(ig, cfg.E, cfg.n_shared, seed=seed)
    widen = functools.partial(synth.widen, dtype="bf16")
    ref = O.lora_moe_layer(xf[toks], io[toks], go[toks], inp["w_gate_up"], inp["w_down"], lora,
                           inp["ws_gate_up"] if cfg.n_shared else None, inp["ws_down"] if cfg.n_shared else None,
                           widen=widen)
    yg = U.y_to_f64(y)[toks]
    err = U.normalized_max_error(yg, ref)
    # the adapters must matter at this size: the same tokens without them are far off
    base = O.moe_layer(xf[toks], io[toks], go[toks], inp["w_gate_up"], inp["w_down"],
                       inp["ws_gate_up"] if cfg.n_shared else None, inp["ws_down"] if cfg.n_shared else None,
                       widen=widen)
    gap = U.normalized_max_error(base, ref)
    U.say(f"  normalised max error {err:.3e} over {len(toks)} tokens, {int(near[toks].sum())} near-ties "
          f"(adapter term {gap:.2e})")
    assert err <= U.BF16_TOL
    assert gap > 3 * U.BF16_TOL
    rel = np.linalg.norm(yg - ref, axis=1) / np.maximum(np.linalg.norm(ref, axis=1), 1e-30)
    assert rel.max() <= 2e-2
    return y


SMALL = [
    # several row tiles per expert with ragged tails; F % 128 = 64 (ragged gate/up column tile)
    synth.LayerConfig("lora_hard", T=600, d=256, F=320, E=8, K=2, route_mode=L.ROUTE_HARD_MASK,
                      mask_set=(0, 2, 5, 7), seed=61),
    synth.LayerConfig("lora_soft", T=700, d=512, F=256, E=8, K=2, route_mode=L.ROUTE_SOFT_PRIOR,
                      mask_set=(0, 2, 5, 7), seed=62),
    synth.LayerConfig("lora_shared_gate_p", T=300, d=256, F=192, E=64, K=6, n_shared=2,
                      route_mode=L.ROUTE_HARD_MASK, gate_mode=L.GATE_P,
                      mask_set=tuple(synth.deepseek_mask_set()), seed=63),
    # few tokens: without adapters this size would take the few-token path
    synth.LayerConfig("lora_three_tokens", T=3, d=256, F=128, E=16, K=4, n_shared=1, route_mode=L.ROUTE_HARD_MASK,
                      gate_mode=L.GATE_P, mask_set=tuple(range(0, 16, 2)), seed=64),
    synth.LayerConfig("lora_plain_k3", T=257, d=128, F=128, E=8, K=3, route_mode=L.ROUTE_PLAIN, seed=65),
]


@pytest.mark.parametrize("cfg", SMALL, ids=lambda c: c.name)
def test_lora_small(cfg):
    check_lora(cfg)


@pytest.mark.parametrize("rank,alpha", [(1, 2.0), (16, 16.0), (12, 24.0)])
def test_lora_ranks(rank, alpha):
    """Rank 1, 12 and 16: one or two 16-column MFMA tiles of the rank projection, padding."""
    check_lora(SMALL[0].with_(name=f"lora_rank{rank}", seed=70 + rank), rank=rank, alpha=alpha)


def test_lora_zero_b_matches_plain_forward_exactly():
    """B = 0 (the adapters' initial state) adds exact zeros in fp32: y is bit-identical to the
    plain forward, which takes the same grouped-GEMM path at this size."""
    cfg = SMALL[0]
    inp = synth.make_layer(cfg)
    lora = synth.make_lora(cfg, 8, 16.0)
    for k in ("b_gate_up", "b_down"):
        lora[k] = np.zeros_like(lora[k])
    y, idx, gate = _run(cfg, inp, lora)
    dd = {k: U.dev(inp[k]) for k in ("x", "w_router", "w_gate_up", "w_down")}
    y0 = L.maskmoe_layer_forward(dd["x"], dd["w_router"], dd["w_gate_up"], dd["w_down"], cfg.K, cfg.route_mode,
                                 cfg.gate_mode, mask=inp["mask"])
    torch.cuda.synchronize()
    assert torch.equal(y, y0)


def test_lora_deterministic_and_dirty_workspace():
    cfg = SMALL[2]
    inp = synth.make_layer(cfg)
    lora = synth.make_lora(cfg)
    desc = L.make_desc(cfg.T, cfg.d, cfg.E, cfg.K, cfg.F, cfg.n_shared, L.BF16, cfg.route_mode, cfg.gate_mode)
    nbytes = L.load().maskmoe_layer_lora_workspace_bytes(desc)
    assert nbytes > L.load().maskmoe_layer_workspace_bytes(desc)
    ws = torch.full((nbytes,), 0xA5, dtype=torch.uint8, device="cuda")
    a, _, _ = _run(cfg, inp, lora, workspace=ws)
    ws.fill_(0x5A)
    b, _, _ = _run(cfg, inp, lora, workspace=ws)
    assert torch.equal(a, b)


def test_lora_empty_tokens():
    cfg = SMALL[0].with_(name="lora_empty", T=0)
    inp = synth.make_layer(cfg)
    y, _, _ = _run(cfg, inp, synth.make_lora(cfg))
    assert y.shape == (0, cfg.d)


def test_lora_rejects_bad_rank():
    cfg = SMALL[4]
    inp = synth.make_layer(cfg)
    with pytest.raises(L.MaskMoEError) as err:
        _run(cfg, inp, synth.make_lora(cfg, 17, 34.0))
    assert err.value.status == L.E_INVAL


def test_lora_mixtral_ft_full_sampled():
    """Mixtral-shaped fine-tuning layer (8192 tokens, d = 4096, F = 14336) with rank-8 adapters."""
    check_lora(synth.mixtral_ft_config(8192), sample=True)
