"""maskmoe_layer_forward_noalloc (the entry point for callers that cannot allocate) against
maskmoe_layer_forward: the same kernels, so the outputs must be bit-identical. Two calls in a
row on one GPU, the second with fewer tokens, so the second runs on the scratch array the
first one left dirty; for the decode path (full Mixtral shape, packed weights, as timed by the
bench) and for the grouped-GEMM path (a small ragged layer with shared experts)."""

import numpy as np
import pytest
import torch

import gpu_util as U
from paper_2609_34077_amd import _lib as L
from paper_2609_34077_amd import synth

pytestmark = pytest.mark.gpu


def _upload(inp, cfg, packed):
    d = {k: U.dev(inp[k]) for k in ("w_router", "w_gate_up", "w_down")}
    d["ws_gate_up"] = U.dev(inp["ws_gate_up"]) if cfg.n_shared else None
    d["ws_down"] = U.dev(inp["ws_down"]) if cfg.n_shared else None
    if packed:
        d["w_gate_up"], d["w_down"] = L.maskmoe_pack_expert_weights(d["w_gate_up"], d["w_down"])
        if cfg.n_shared:
            d["ws_gate_up"], d["ws_down"] = L.maskmoe_pack_expert_weights(d["ws_gate_up"], d["ws_down"])
    return d


def _both(cfg, inp, dd, x, packed):
    mp = dict(mask=inp["mask"]) if cfg.route_mode == L.ROUTE_HARD_MASK else dict(prior=inp["prior"])
    T = x.shape[0]
    lay = L.LAYOUT_PACKED if packed else L.LAYOUT_ROWS
    out = []
    for fn in ("plain", "noalloc"):
        y = torch.empty((T, cfg.d), dtype=torch.bfloat16, device="cuda")
        idx = torch.empty((T, cfg.K), dtype=torch.int32, device="cuda")
        gate = torch.empty((T, cfg.K), dtype=torch.float32, device="cuda")
        kw = dict(ws_gate_up=dd["ws_gate_up"], ws_down=dd["ws_down"], topk_idx=idx, topk_gate=gate,
                  weight_layout=lay, **mp)
        if fn == "plain":
            L.maskmoe_layer_forward(x, dd["w_router"], dd["w_gate_up"], dd["w_down"], cfg.K, cfg.route_mode,
                                    cfg.gate_mode, y=y, **kw)
        else:
            L.maskmoe_layer_forward_noalloc(x, dd["w_router"], dd["w_gate_up"], dd["w_down"], cfg.K,
                                            cfg.route_mode, cfg.gate_mode, y, **kw)
        torch.cuda.synchronize()
        out.append((y, idx, gate))
    (y0, i0, g0), (y1, i1, g1) = out
    assert torch.equal(i0, i1) and torch.equal(g0, g1)
    assert torch.equal(y0.view(torch.int16), y1.view(torch.int16))


CASES = [
    # decode path at the full Mixtral shape, packed weights: 16 tokens, then 4
    (synth.mixtral_decode_config(16), True, (16, 4)),
    # grouped-GEMM path, shared experts, ragged tiles: 300 tokens, then 40
    (synth.LayerConfig("noalloc_shared", T=300, d=256, F=192, E=64, K=6, n_shared=2,
                       route_mode=L.ROUTE_HARD_MASK, gate_mode=L.GATE_P,
                       mask_set=tuple(synth.deepseek_mask_set()), seed=91), False, (300, 40)),
]


@pytest.mark.parametrize("cfg,packed,sizes", CASES, ids=lambda c: getattr(c, "name", None))
def test_noalloc_matches_layer_forward_two_calls(cfg, packed, sizes):
    U.say(f"noalloc vs layer forward: {cfg.name}, token counts {sizes}")
    inp = synth.make_layer(cfg)
    dd = _upload(inp, cfg, packed)
    x_all = U.dev(inp["x"])
    for T in sizes:
        _both(cfg, inp, dd, x_all[:T].contiguous(), packed)


def test_noalloc_rejects_sizes_beyond_its_scratch():
    x = torch.zeros((8192, 64), dtype=torch.bfloat16, device="cuda")
    w = torch.zeros((8, 64), dtype=torch.bfloat16, device="cuda")
    gu = torch.zeros((8, 2 * 14336, 64), dtype=torch.bfloat16, device="cuda")
    dn = torch.zeros((8, 64, 14336), dtype=torch.bfloat16, device="cuda")
    y = torch.empty((8192, 64), dtype=torch.bfloat16, device="cuda")
    desc = L.make_desc(8192, 64, 8, 2, 14336, 0, L.BF16, L.ROUTE_PLAIN, L.GATE_RENORM)
    assert L.maskmoe_layer_workspace_bytes(desc) > L.NOALLOC_SCRATCH_BYTES
    with pytest.raises(L.MaskMoEError) as err:
        L.maskmoe_layer_forward_noalloc(x, w, gu, dn, 2, L.ROUTE_PLAIN, L.GATE_RENORM, y)
    assert err.value.status == L.E_WORKSPACE
