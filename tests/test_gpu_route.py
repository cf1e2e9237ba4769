"""GPU parity of maskmoe_route against the oracle (Section 3.1 Eq. 1, Eq. 2, Eq. 4)."""

import numpy as np
import pytest
import torch

import gpu_util as U
from oracle import routing as R
from paper_2609_34077_amd import _lib as L
from paper_2609_34077_amd import synth

pytestmark = pytest.mark.gpu


def _inputs(T, d, E, dtype, seed, Lyr=None):
    g = np.random.default_rng(seed)
    shape_w = (E, d) if Lyr is None else (Lyr, E, d)
    x = g.standard_normal((T, d)).astype(np.float32)
    w = (0.02 * g.standard_normal(shape_w)).astype(np.float32)
    if dtype == "bf16":
        return synth.bf16_bits(x), synth.bf16_bits(w)
    return x, w


def _run_and_check(T, d, E, K, mode, gate_mode, dtype, seed, mask=None, prior=None, max_near_frac=0.05):
    U.say(f"route T={T} d={d} E={E} K={K} mode={mode} gate={gate_mode} {dtype} seed={seed}")
    x, w = _inputs(T, d, E, dtype, seed)
    idx, gate, margin = L.maskmoe_route(U.dev(x), U.dev(w), K, mode, gate_mode, mask=mask, prior=prior)
    torch.cuda.synchronize()
    z = R.router_logits(U.f64(x, dtype), U.f64(w, dtype))
    near = U.check_routing(z, idx.cpu().numpy(), gate.cpu().numpy(), margin.cpu().numpy(), K, mode,
                           gate_mode, mask, prior)
    assert near <= max(2, int(T * max_near_frac))
    U.say(f"  near-tie tokens {near} of {T}")
    return idx, gate, margin


MODES = [(L.ROUTE_PLAIN, None), (L.ROUTE_HARD_MASK, "mask"), (L.ROUTE_SOFT_PRIOR, "prior")]


def _mp(kind, E, keep, delta=1.0):
    if kind == "mask":
        return dict(mask=synth.binary_mask(E, keep))
    if kind == "prior":
        return dict(prior=synth.concentrated_prior(E, keep, delta))
    return {}


@pytest.mark.parametrize("mode,kind", MODES)
@pytest.mark.parametrize("gate_mode", [L.GATE_P, L.GATE_RENORM])
def test_tiny_f32(mode, kind, gate_mode):
    _run_and_check(64, 256, 8, 2, mode, gate_mode, "f32", 0, **_mp(kind, 8, [0, 2, 5, 7]))


@pytest.mark.parametrize("T", [1, 4, 16, 17, 129, 1000])
@pytest.mark.parametrize("mode,kind", MODES)
def test_mixtral_shaped(T, mode, kind):
    _run_and_check(T, 4096, 8, 2, mode, L.GATE_RENORM, "bf16", T, **_mp(kind, 8, [0, 2, 5, 7]))


@pytest.mark.parametrize("T", [3, 333])
@pytest.mark.parametrize("mode,kind", MODES)
def test_deepseek_shaped(T, mode, kind):
    _run_and_check(T, 2048, 64, 6, mode, L.GATE_P, "bf16", 100 + T, **_mp(kind, 64, synth.deepseek_mask_set()))


@pytest.mark.parametrize("E,K,T", [(256, 16, 70), (256, 1, 200), (16, 16, 40), (5, 3, 33), (1, 1, 9)])
def test_extreme_expert_counts(E, K, T):
    # 256 experts with d = 128 put many keys within 1e-3 of each other: near-ties are common
    _run_and_check(T, 128, E, K, L.ROUTE_SOFT_PRIOR, L.GATE_RENORM, "bf16", E * 31 + K,
                   prior=synth.concentrated_prior(E, list(range(0, E, 3)), 0.7), max_near_frac=0.6)


@pytest.mark.parametrize("T", [5, 300])
def test_multi_layer_trace_router(T):
    Lyr, E, K, d = 32, 8, 2, 4096
    U.say(f"route multi-layer L={Lyr} T={T}")
    x, w = _inputs(T, d, E, "bf16", 77 + T, Lyr=Lyr)
    cfg = synth.TraceConfig(L=Lyr)
    sets = synth.trace_layer_sets(cfg)
    prior = np.stack([synth.concentrated_prior(E, s, 1.0) for s in sets])
    idx, gate, margin = L.maskmoe_route(U.dev(x), U.dev(w), K, L.ROUTE_SOFT_PRIOR, L.GATE_RENORM, prior=prior)
    torch.cuda.synchronize()
    xf = U.f64(x, "bf16")
    wf = U.f64(w, "bf16")
    idx, gate, margin = idx.cpu().numpy(), gate.cpu().numpy(), margin.cpu().numpy()
    for l in range(Lyr):
        z = R.router_logits(xf, wf[l])
        U.check_routing(z, idx[l], gate[l], margin[l], K, L.ROUTE_SOFT_PRIOR, L.GATE_RENORM, prior=prior[l])


# Many tokens x many router outputs: the LDS-tiled router GEMM path. Ragged token tiles, a
# second block of layers (40 x 8 outputs), a 240-output tile (E = 48), and E = 256.
ROUTE_GEMM_CASES = [
    (1100, 4096, 8, 2, 32, L.ROUTE_SOFT_PRIOR, L.GATE_RENORM),
    (1024, 256, 8, 2, 40, L.ROUTE_HARD_MASK, L.GATE_RENORM),
    (1500, 512, 64, 6, 4, L.ROUTE_SOFT_PRIOR, L.GATE_P),
    (1030, 192, 48, 4, 5, L.ROUTE_PLAIN, L.GATE_RENORM),
    (1024, 128, 256, 16, 1, L.ROUTE_HARD_MASK, L.GATE_P),
]


@pytest.mark.parametrize("T,d,E,K,Lyr,mode,gate_mode", ROUTE_GEMM_CASES,
                         ids=lambda v: str(v))
def test_many_tokens_many_layers(T, d, E, K, Lyr, mode, gate_mode):
    U.say(f"route gemm path T={T} d={d} E={E} K={K} L={Lyr} mode={mode} gate={gate_mode}")
    x, w = _inputs(T, d, E, "bf16", 1000 + T + Lyr, Lyr=Lyr)
    rng = np.random.default_rng(T + E)
    keep = [sorted(rng.choice(E, max(K, E // 2), replace=False)) for _ in range(Lyr)]
    mask = np.stack([synth.binary_mask(E, k) for k in keep]) if mode == L.ROUTE_HARD_MASK else None
    prior = np.stack([synth.concentrated_prior(E, k, 1.0) for k in keep]) if mode == L.ROUTE_SOFT_PRIOR else None
    idx, gate, margin = L.maskmoe_route(U.dev(x), U.dev(w), K, mode, gate_mode, mask=mask, prior=prior)
    torch.cuda.synchronize()
    xf, wf = U.f64(x, "bf16"), U.f64(w, "bf16")
    idx, gate, margin = idx.cpu().numpy(), gate.cpu().numpy(), margin.cpu().numpy()
    near = 0
    for l in range(Lyr):
        near += U.check_routing(R.router_logits(xf, wf[l]), idx[l], gate[l], margin[l], K, mode, gate_mode,
                                None if mask is None else mask[l], None if prior is None else prior[l])
    U.say(f"  near-tie (token, layer) pairs {near} of {T * Lyr}")
    assert near <= max(2, int(T * Lyr * (0.6 if E == 256 else 0.05)))


def test_mode_equivalences_bit_exact():
    T, d, E, K = 500, 1024, 8, 2
    x, w = _inputs(T, d, E, "bf16", 5)
    xd, wd = U.dev(x), U.dev(w)
    ip, gp, mp = L.maskmoe_route(xd, wd, K, L.ROUTE_PLAIN, L.GATE_RENORM)
    ih, gh, mh = L.maskmoe_route(xd, wd, K, L.ROUTE_HARD_MASK, L.GATE_RENORM, mask=np.ones(E, np.uint8))
    iu, gu, mu = L.maskmoe_route(xd, wd, K, L.ROUTE_SOFT_PRIOR, L.GATE_RENORM, prior=np.full(E, 0.125, np.float32))
    assert torch.equal(ip, ih) and torch.equal(gp, gh) and torch.equal(mp, mh)
    # a uniform prior shifts every key by the same constant: same order up to sub-ulp ties
    assert torch.equal(ip, iu) and torch.equal(gp, gu)
    keep = [1, 6]
    ik, gk, mk = L.maskmoe_route(xd, wd, K, L.ROUTE_HARD_MASK, L.GATE_RENORM, mask=synth.binary_mask(E, keep))
    assert (ik.sort(dim=1).values.cpu() == torch.tensor(keep, dtype=torch.int32)).all()
    assert torch.isinf(mk).all()


def test_deterministic_repeat():
    x, w = _inputs(777, 2048, 64, "bf16", 9)
    xd, wd = U.dev(x), U.dev(w)
    prior = synth.concentrated_prior(64, synth.deepseek_mask_set(), 1.0)
    a = L.maskmoe_route(xd, wd, 6, L.ROUTE_SOFT_PRIOR, L.GATE_P, prior=prior)
    b = L.maskmoe_route(xd, wd, 6, L.ROUTE_SOFT_PRIOR, L.GATE_P, prior=prior)
    for u, v in zip(a, b):
        assert torch.equal(u, v)


def test_empty_tokens():
    x = torch.empty((0, 64), dtype=torch.bfloat16, device="cuda")
    w = torch.zeros((8, 64), dtype=torch.bfloat16, device="cuda")
    idx, gate, margin = L.maskmoe_route(x, w, 2, L.ROUTE_PLAIN, L.GATE_RENORM)
    assert idx.shape == (0, 2)


def test_full_trace_router_sampled():
    """Routing-and-fetch trace router at full size (32 layers, 131072 AR(1) tokens); the
    oracle checks a random sample of 1024 tokens in every layer."""
    cfg = synth.TraceConfig()
    U.say("route full trace: generating AR(1) inputs")
    inp = synth.make_trace_inputs(cfg)
    xd, wd = U.dev(inp["x"]), U.dev(inp["w_router"])
    U.say("route full trace: running")
    idx, gate, margin = L.maskmoe_route(xd, wd, cfg.K, L.ROUTE_SOFT_PRIOR, L.GATE_RENORM, prior=inp["prior"])
    torch.cuda.synchronize()
    sample = np.sort(np.random.default_rng(3).choice(cfg.S * cfg.N, 1024, replace=False))
    xs = U.f64(inp["x"][sample], "bf16")
    ws = U.f64(inp["w_router"], "bf16")
    sd = torch.from_numpy(sample).cuda()
    ig, gg, mg = idx[:, sd].cpu().numpy(), gate[:, sd].cpu().numpy(), margin[:, sd].cpu().numpy()
    for l in range(cfg.L):
        U.check_routing(R.router_logits(xs, ws[l]), ig[l], gg[l], mg[l], cfg.K, L.ROUTE_SOFT_PRIOR,
                        L.GATE_RENORM, prior=inp["prior"][l])
    # properties at every token: distinct in-range experts, renormalised gates sum to 1
    ia = idx.cpu().numpy()
    assert ((ia >= 0) & (ia < cfg.E)).all() and (ia[..., 0] != ia[..., 1]).all()
    np.testing.assert_allclose(gate.sum(-1).cpu().numpy(), 1.0, atol=1e-5)


# Split routing (logits to a workspace, then a selection kernel) against the one-kernel
# routing: the same bits in idx, gate and margin. Router GEMM path and small-tile path; one
# thread per pair (E <= 16, E % 4 != 0 included) and one wavefront per pair (16 < E <= 64).
SPLIT_CASES = [
    (1100, 4096, 8, 2, 32, L.ROUTE_SOFT_PRIOR, L.GATE_RENORM),
    (1500, 512, 64, 6, 4, L.ROUTE_SOFT_PRIOR, L.GATE_P),
    (1030, 192, 48, 4, 5, L.ROUTE_PLAIN, L.GATE_RENORM),
    (1024, 256, 16, 16, 8, L.ROUTE_HARD_MASK, L.GATE_P),
    (2000, 2048, 64, 6, 1, L.ROUTE_HARD_MASK, L.GATE_P),
    (600, 4096, 8, 2, 1, L.ROUTE_SOFT_PRIOR, L.GATE_RENORM),
    (700, 256, 17, 3, 1, L.ROUTE_SOFT_PRIOR, L.GATE_RENORM),
    (515, 128, 5, 3, 3, L.ROUTE_HARD_MASK, L.GATE_P),
    (512, 64, 64, 16, 1, L.ROUTE_PLAIN, L.GATE_RENORM),
    # softmax over all E (g = p) with 16 < E < 64: the normaliser's pairwise tree with experts
    # past E counting as 0, on both the wavefront and the per-thread selection
    (640, 256, 17, 2, 1, L.ROUTE_SOFT_PRIOR, L.GATE_P),
    (520, 128, 48, 6, 2, L.ROUTE_PLAIN, L.GATE_P),
    (1030, 192, 40, 4, 3, L.ROUTE_HARD_MASK, L.GATE_P),
]


def _bits(t):
    return t.contiguous().view(torch.int32).cpu()


@pytest.mark.parametrize("T,d,E,K,Lyr,mode,gate_mode", SPLIT_CASES, ids=lambda v: str(v))
def test_split_routing_matches_fused_bitwise(T, d, E, K, Lyr, mode, gate_mode):
    U.say(f"route split vs fused T={T} d={d} E={E} K={K} L={Lyr} mode={mode} gate={gate_mode}")
    x, w = _inputs(T, d, E, "bf16", 4000 + T + E, Lyr=Lyr)
    rng = np.random.default_rng(T * E)
    keep = [sorted(rng.choice(E, max(K, E // 2), replace=False)) for _ in range(Lyr)]
    mask = np.stack([synth.binary_mask(E, k) for k in keep]) if mode == L.ROUTE_HARD_MASK else None
    prior = np.stack([synth.concentrated_prior(E, k, 1.0) for k in keep]) if mode == L.ROUTE_SOFT_PRIOR else None
    xd, wd = U.dev(x), U.dev(w)
    desc = L.make_desc(T, d, E, K, dtype=L.BF16, route_mode=mode, gate_mode=gate_mode)
    nbytes = L.load().maskmoe_route_workspace_bytes(desc, Lyr)
    assert nbytes == Lyr * T * E * 4
    ws = torch.full((nbytes,), 0x7F, dtype=torch.uint8, device="cuda")
    a = L.maskmoe_route(xd, wd, K, mode, gate_mode, mask=mask, prior=prior, workspace=ws)
    b = L.maskmoe_route(xd, wd, K, mode, gate_mode, mask=mask, prior=prior, workspace=None)
    torch.cuda.synchronize()
    assert torch.equal(a[0], b[0])
    assert torch.equal(_bits(a[1]), _bits(b[1])) and torch.equal(_bits(a[2]), _bits(b[2]))
    # the split logits are the router logits (fp32 accumulation of the bf16 products)
    z = ws.view(torch.float32).view(Lyr, T, E).cpu().double().numpy()
    zr = np.stack([R.router_logits(U.f64(x, "bf16")[:64], U.f64(w, "bf16").reshape(Lyr, E, d)[l]) for l in range(Lyr)])
    np.testing.assert_allclose(z[:, :64], zr, rtol=1e-4, atol=1e-4 * np.abs(zr).max())


def test_split_routing_non_finite_logits_match_fused():
    """Tokens whose logits are all NaN, or +inf / -inf for some experts: the fallback picks
    (lowest untaken index) and the NaN / inf gates of both paths carry the same bits."""
    T, d, E, K = 640, 128, 32, 4
    x, w = _inputs(T, d, E, "bf16", 91)
    xt = torch.from_numpy(x).view(torch.bfloat16).clone()
    xt[3] = float("nan")
    xt[100, 0] = float("inf")
    xt[101, 5] = float("-inf")
    xd = xt.cuda()
    wd = U.dev(w)
    for mode, gm, kw in [(L.ROUTE_PLAIN, L.GATE_RENORM, {}), (L.ROUTE_SOFT_PRIOR, L.GATE_P,
                                                            dict(prior=synth.concentrated_prior(E, [1, 2, 9], 1.0)))]:
        a = L.maskmoe_route(xd, wd, K, mode, gm, workspace="auto", **kw)
        b = L.maskmoe_route(xd, wd, K, mode, gm, workspace=None, **kw)
        torch.cuda.synchronize()
        assert torch.equal(a[0], b[0])
        assert torch.equal(_bits(a[1]), _bits(b[1])) and torch.equal(_bits(a[2]), _bits(b[2]))
        assert a[0][3].tolist() == list(range(K))   # every key NaN: the lowest indices
