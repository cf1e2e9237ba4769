"""GPU parity of maskmoe_cache_fetches against the oracle LRU (Section 4.1, Eq. 5); bit-exact."""

import numpy as np
import pytest
import torch

import gpu_util as U
from conftest import golden_path
from oracle import cache as C
from oracle import routing as R
from paper_2609_34077_amd import _lib as L
from paper_2609_34077_amd import synth

pytestmark = pytest.mark.gpu


def _gpu(trace, E, B, state=None, fps=True, policy=L.CACHE_LRU, counts=None):
    st = None if state is None else torch.from_numpy(np.ascontiguousarray(state, dtype=np.int32)).cuda()
    ct = None if counts is None else torch.from_numpy(np.ascontiguousarray(counts, dtype=np.int32)).cuda()
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    out = L.maskmoe_cache_fetches(torch.from_numpy(np.ascontiguousarray(trace, dtype=np.int32)).cuda(), E, B,
                                  state=st, with_f_per_step=fps, dev_error=err, policy=policy, counts=ct)
    torch.cuda.synchronize()
    res = {k: (v.cpu().numpy() if v is not None else None) for k, v in out.items()}
    res["state"] = None if st is None else st.cpu().numpy()
    res["counts"] = None if ct is None else ct.cpu().numpy()
    return res


def _compare(trace, E, B, state=None, policy=L.CACHE_LRU, counts=None):
    g = _gpu(trace, E, B, state, policy=policy, counts=counts)
    out = C.cache_fetches(trace, E, B, state, policy=policy, counts=counts)
    f, h, fps, final, bad = out[:5]
    np.testing.assert_array_equal(g["fetches"], f)
    np.testing.assert_array_equal(g["hits"], h)
    np.testing.assert_array_equal(g["f_per_step"], fps)
    assert int(g["dev_error"][0]) == int(bad)
    if state is not None:
        np.testing.assert_array_equal(g["state"], final)
    if counts is not None and policy == L.CACHE_LFU:
        np.testing.assert_array_equal(g["counts"], out[5])
    return g


def test_hand_trace():
    steps = [[0, 1], [2, 3], [4, 5], [2, 6], [2, 7], [0, 5], [2, 3], [1, 5]]
    tr = np.array(steps, np.int32)[None, None]
    state = np.full((1, 1, 4), -1, np.int32)
    g = _compare(tr, 8, 4, state)
    assert g["f_per_step"][0, 0].tolist() == [2, 2, 2, 1, 1, 1, 1, 1]
    assert g["state"][0, 0].tolist() == [2, 3, 5, 1]
    assert int(_gpu(tr, 8, 2)["fetches"][0, 0]) == 15
    assert int(_gpu(tr, 8, 8)["fetches"][0, 0]) == 8


@pytest.mark.parametrize("E,K,B,N", [(8, 2, 4, 512), (8, 2, 2, 100), (8, 2, 7, 65), (8, 2, 8, 33),
                                     (8, 2, 20, 40), (64, 6, 12, 300), (64, 6, 6, 77), (16, 3, 5, 1),
                                     (33, 11, 32, 50), (64, 64, 64, 10), (5, 1, 1, 200),
                                     # several 512-step chunks with a ragged last one; 9..16 experts
                                     (8, 2, 4, 1100), (12, 3, 5, 600), (9, 4, 4, 513), (16, 16, 16, 30),
                                     (17, 2, 4, 520)])
def test_random_traces_bit_exact(E, K, B, N):
    U.say(f"cache E={E} K={K} B={B} N={N}")
    tr = synth.random_trace(3, 7, N, K, E, seed=E * 1000 + B * 10 + K, locality=0.6)
    _compare(tr, E, B)
    st = np.full((3, 7, B), -1, np.int32)
    _compare(tr, E, B, st)


def test_initial_state_and_resume():
    E, K, B = 8, 2, 4
    tr = synth.random_trace(2, 5, 200, K, E, seed=11, locality=0.5)
    whole = _gpu(tr, E, B, np.full((2, 5, B), -1, np.int32))
    first = _gpu(tr[:, :, :77], E, B, np.full((2, 5, B), -1, np.int32))
    second = _gpu(tr[:, :, 77:], E, B, first["state"])
    np.testing.assert_array_equal(whole["fetches"], first["fetches"] + second["fetches"])
    np.testing.assert_array_equal(whole["f_per_step"], np.concatenate([first["f_per_step"], second["f_per_step"]], 2))
    np.testing.assert_array_equal(whole["state"], second["state"])
    # a non-empty, partly filled initial state
    st = np.full((2, 5, B), -1, np.int32)
    st[:, :, 0] = 3
    st[:, :, 1] = 6
    _compare(tr, E, B, st)


def test_invalid_entries_flagged_and_skipped():
    tr = np.array([[[[0, 9], [1, 1], [-1, 2], [3, 4]]]], np.int32)
    g = _compare(tr, 8, 4)
    assert int(g["dev_error"][0]) == 1
    assert g["f_per_step"][0, 0].tolist() == [1, 1, 1, 2]


def test_empty_trace_steps():
    tr = np.zeros((2, 3, 0, 2), np.int32)
    g = _gpu(tr, 8, 4, np.full((2, 3, 4), -1, np.int32), fps=False)
    assert (g["fetches"] == 0).all() and (g["hits"] == 0).all()


def test_full_size_trace_sampled_streams():
    """[32 layers, 256 streams, 512 steps, K=2] with B=4; the oracle replays 400 random streams."""
    Lyr, S, N, K, E, B = 32, 256, 512, 2, 8, 4
    U.say("cache full size: building trace")
    g = np.random.default_rng(0)
    # sticky random trace, generated vectorised: keep the previous pair with prob. 0.7
    tr = np.empty((Lyr, S, N, K), np.int32)
    pair = np.stack([g.permutation(E)[:K] for _ in range(Lyr * S)]).reshape(Lyr, S, K)
    for n in range(N):
        redraw = g.random((Lyr, S)) > 0.7
        fresh = np.argsort(g.random((Lyr, S, E)), axis=-1)[..., :K].astype(np.int32)
        pair = np.where(redraw[..., None], fresh, pair)
        tr[:, :, n] = pair
    res = _gpu(tr, E, B)
    assert int(res["dev_error"][0]) == 0
    picks = g.choice(Lyr * S, 400, replace=False)
    for p in picks:
        l, s = divmod(int(p), S)
        f, h, _, _ = C.lru_stream(tr[l, s].tolist(), E, B)
        assert res["fetches"][l, s] == sum(f) and res["hits"][l, s] == sum(h)
        assert res["f_per_step"][l, s].tolist() == f
    assert (res["fetches"] + res["hits"] == N * K).all()


@pytest.mark.parametrize("delta", [1.0, 0.0])
def test_route_then_replay_end_to_end(delta):
    """Trace workload at reduced size: GPU routing -> GPU cache vs oracle routing -> oracle cache.

    Streams whose tokens all have a clear margin must agree bit-exactly; a stream with a
    near-tie must still replay the oracle's own trace bit-exactly on the GPU.
    """
    cfg = synth.TraceConfig(S=24, N=160)
    inp = synth.make_trace_inputs(cfg)
    prior = inp["prior"] if delta else inp["prior_zero"]
    xd, wd = U.dev(inp["x"]), U.dev(inp["w_router"])
    idx, _, _ = L.maskmoe_route(xd, wd, cfg.K, L.ROUTE_SOFT_PRIOR, L.GATE_RENORM, prior=prior)
    trace_g = idx.view(cfg.L, cfg.S, cfg.N, cfg.K)
    res = L.maskmoe_cache_fetches(trace_g, cfg.E, cfg.B)
    torch.cuda.synchronize()
    xf, wf = U.f64(inp["x"], "bf16"), U.f64(inp["w_router"], "bf16")
    io, go, mo = R.route_layers(xf, wf, cfg.K, R.SOFT_PRIOR, R.GATE_RENORM, priors=prior)
    trace_o = io.reshape(cfg.L, cfg.S, cfg.N, cfg.K).astype(np.int32)
    f_o, h_o, _, _, _ = C.cache_fetches(trace_o, cfg.E, cfg.B)
    clear = (mo.reshape(cfg.L, cfg.S, cfg.N) > U.MARGIN_TOL).all(axis=2)
    tg = np.sort(trace_g.cpu().numpy(), axis=-1)
    same = (tg == np.sort(trace_o, axis=-1)).all(axis=(2, 3))
    assert same[clear].all()          # clear streams route identically
    fg = res["fetches"].cpu().numpy()
    np.testing.assert_array_equal(fg[same], f_o[same])
    U.say(f"  streams: {clear.sum()} all-clear, {same.sum()} identical traces of {clear.size}")
    assert same.sum() >= clear.sum() > 0
    # the GPU cache on the oracle's trace is bit-exact everywhere
    g2 = _gpu(trace_o, cfg.E, cfg.B)
    np.testing.assert_array_equal(g2["fetches"], f_o)
    np.testing.assert_array_equal(g2["hits"], h_o)


def _trace_inputs_full():
    if "full" not in _TRACE_CACHE:
        U.say("trace full size: generating AR(1) inputs (256 sequences x 512 steps, d = 4096)")
        cfg = synth.TraceConfig()
        _TRACE_CACHE["full"] = (cfg, synth.make_trace_inputs(cfg))
    return _TRACE_CACHE["full"]


_TRACE_CACHE = {}


@pytest.mark.parametrize("delta", [1.0, 0.0])
def test_trace_full_size_fetch_parity(delta):
    """The routing-and-fetch trace at full size (32 layers, 256 sequences x 512 AR(1) steps,
    K = 2, LRU with B = 4, each (layer, sequence) its own cache starting empty), with the
    per-layer prior and with the zero prior (Eq. 4; Eq. 5's counts).

    The GPU routes all 131072 tokens through the 32 routers (maskmoe_route, split routing) and
    replays the whole trace (maskmoe_cache_fetches). The oracle routes every token in float64;
    where its margin is <= 1e-3 it adopts the GPU's set after checking it is a valid Top-K
    (gpu_util.effective_routing), and replays every stream in Python. Fetches and hits must be
    bit-exact for all 8192 (layer, sequence) streams, and so must Fetches/tok (Eq. 5).
    """
    cfg, inp = _trace_inputs_full()
    prior = inp["prior"] if delta else inp["prior_zero"]
    U.say(f"trace full size, delta={delta}: GPU routing + cache replay")
    xd, wd = U.dev(inp["x"]), U.dev(inp["w_router"])
    idx, _, _ = L.maskmoe_route(xd, wd, cfg.K, L.ROUTE_SOFT_PRIOR, L.GATE_RENORM, prior=prior, with_margin=False)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    res = L.maskmoe_cache_fetches(idx.view(cfg.L, cfg.S, cfg.N, cfg.K), cfg.E, cfg.B, dev_error=err)
    torch.cuda.synchronize()
    ig = idx.cpu().numpy()                       # [L, S*N, K]
    fg, hg = res["fetches"].cpu().numpy(), res["hits"].cpu().numpy()
    assert int(err.item()) == 0
    del xd, wd, idx
    T = cfg.S * cfg.N
    if "z" not in _TRACE_CACHE:   # the logits do not depend on the prior
        U.say("  oracle router logits (float64) of every token through the 32 routers")
        wf = U.f64(inp["w_router"], "bf16").reshape(cfg.L * cfg.E, cfg.d)
        z = np.empty((cfg.L, T, cfg.E))
        step = 16384
        for t0 in range(0, T, step):
            zc = R.router_logits(U.f64(inp["x"][t0:t0 + step], "bf16"), wf)   # [t, L*E]
            z[:, t0:t0 + step] = zc.reshape(-1, cfg.L, cfg.E).transpose(1, 0, 2)
        _TRACE_CACHE["z"] = z
    z = _TRACE_CACHE["z"]
    trace_o = np.empty((cfg.L, T, cfg.K), np.int32)
    near_total = clear_streams = 0
    for l in range(cfg.L):
        io, _, near = U.effective_routing(z[l], ig[l], cfg.K, R.SOFT_PRIOR, R.GATE_RENORM, prior=prior[l])
        trace_o[l] = io
        near_total += int(near.sum())
        clear_streams += int((~near.reshape(cfg.S, cfg.N).any(axis=1)).sum())
    U.say(f"  near-tie (layer, token) pairs {near_total} of {cfg.L * T} (GPU set adopted after validation); "
          f"{clear_streams} of {cfg.L * cfg.S} streams have no near-tie")
    assert clear_streams >= 32
    U.say("  oracle cache replay of all 8192 streams")
    f_o, h_o, _, _, bad = C.cache_fetches(trace_o.reshape(cfg.L, cfg.S, cfg.N, cfg.K), cfg.E, cfg.B)
    assert not bad
    np.testing.assert_array_equal(fg, f_o)
    np.testing.assert_array_equal(hg, h_o)
    fpt = C.fetches_per_token(int(f_o.sum()), T)
    U.say(f"  Fetches/tok {fpt:.4f} (delta={delta}), bit-exact on every (layer, sequence)")
    assert 0 < fpt <= cfg.L * cfg.K


POLICIES = [L.CACHE_LRU, L.CACHE_LFU, L.CACHE_FIFO]


@pytest.mark.parametrize("policy", POLICIES)
@pytest.mark.parametrize("E,K,B,N", [(8, 2, 4, 300), (8, 2, 3, 65), (64, 6, 12, 200), (16, 3, 16, 40),
                                     (6, 1, 2, 130), (64, 64, 64, 5), (12, 2, 4, 700), (16, 4, 6, 1030)])
def test_policies_bit_exact(policy, E, K, B, N):
    U.say(f"cache policy={policy} E={E} K={K} B={B} N={N}")
    tr = synth.random_trace(2, 9, N, K, E, seed=E * 31 + B * 7 + K + policy, locality=0.55)
    _compare(tr, E, B, policy=policy)
    st = np.full((2, 9, B), -1, np.int32)
    cnt = np.random.default_rng(policy).integers(0, 5, size=(2, 9, E)).astype(np.int32)
    _compare(tr, E, B, st, policy=policy, counts=cnt)


def test_policy_hand_traces():
    steps = [[0, 1], [2, 3], [4, 5], [2, 6], [2, 7], [0, 5], [2, 3], [1, 5]]
    tr = np.array(steps, np.int32)[None, None]
    for policy, total, final in ((L.CACHE_FIFO, 13, [2, 3, 1, 5]), (L.CACHE_LFU, 11, [2, 3, 5, 1])):
        g = _compare(tr, 8, 4, np.full((1, 1, 4), -1, np.int32), policy=policy, counts=np.zeros((1, 1, 8), np.int32))
        assert int(g["fetches"][0, 0]) == total and g["state"][0, 0].tolist() == final
    tr2 = np.array([0, 0, 0, 1, 2, 0], np.int32).reshape(1, 1, 6, 1)
    for policy, fexp in ((L.CACHE_LRU, [1, 0, 0, 1, 1, 1]), (L.CACHE_FIFO, [1, 0, 0, 1, 1, 1]),
                         (L.CACHE_LFU, [1, 0, 0, 1, 1, 0])):
        g = _compare(tr2, 3, 2, policy=policy)
        assert g["f_per_step"][0, 0].tolist() == fexp


@pytest.mark.parametrize("policy", [L.CACHE_LFU, L.CACHE_FIFO])
def test_resume_with_state_and_counts(policy):
    E, K, B = 8, 2, 4
    tr = synth.random_trace(2, 5, 200, K, E, seed=12 + policy, locality=0.5)
    z = lambda: (np.full((2, 5, B), -1, np.int32), np.zeros((2, 5, E), np.int32))
    s0, c0 = z()
    whole = _gpu(tr, E, B, s0, policy=policy, counts=c0)
    s1, c1 = z()
    first = _gpu(tr[:, :, :61], E, B, s1, policy=policy, counts=c1)
    second = _gpu(tr[:, :, 61:], E, B, first["state"], policy=policy, counts=first["counts"])
    np.testing.assert_array_equal(whole["fetches"], first["fetches"] + second["fetches"])
    np.testing.assert_array_equal(whole["state"], second["state"])
    np.testing.assert_array_equal(whole["counts"], second["counts"])


@pytest.mark.parametrize("E", [8, 12, 20])
def test_invalid_initial_state_entries_skipped_and_flagged(E):
    """Initial states listing an expert twice or an index >= E: those entries are skipped (the
    oracle's reading of the state) and the device error flag is raised."""
    K, B = 2, 4
    tr = synth.random_trace(2, 5, 90, K, E, seed=E + 5, locality=0.5)
    st = np.full((2, 5, B), -1, np.int32)
    st[:, :, 0], st[:, :, 1], st[:, :, 2] = 3, 3, E + 1
    st[1, 2] = [5, -1, 1, E]
    g = _gpu(tr, E, B, st)
    f, h, fps, final, bad = C.cache_fetches(tr, E, B, st)[:5]
    np.testing.assert_array_equal(g["fetches"], f)
    np.testing.assert_array_equal(g["hits"], h)
    np.testing.assert_array_equal(g["f_per_step"], fps)
    np.testing.assert_array_equal(g["state"], final)
    assert not bad and int(g["dev_error"][0]) == 1


@pytest.mark.parametrize("policy", POLICIES)
def test_long_persistent_streams(policy):
    """Caches kept across sequences: 3 layers x 1 stream of 131072 steps (the trace workload's
    sequences back to back), E = 8, K = 2, B = 4; every step against the oracle."""
    Lyr, N, K, E, B = 3, 131072, 2, 8, 4
    U.say(f"cache persistent streams policy={policy} N={N}")
    tr = synth.random_trace(Lyr, 1, N, K, E, seed=77 + policy, locality=0.6)
    _compare(tr, E, B, policy=policy)


@pytest.mark.parametrize("E", [8, 12])
def test_invalid_entries_long_trace(E):
    """Invalid entries (negative, >= E, repeated within a step) in traces long enough for the
    several-streams-per-wavefront kernel: skipped and flagged as the oracle does."""
    tr = synth.random_trace(2, 9, 300, 3, E, seed=E * 7, locality=0.5)
    tr[0, 1, 5] = [1, 1, 2]
    tr[1, 8, 299] = [-1, 0, 3]
    tr[1, 0, 70] = [E, E + 5, 2]
    g = _compare(tr, E, 4)
    assert int(g["dev_error"][0]) == 1
    assert g["f_per_step"][0, 1, 5] <= 2 and g["f_per_step"][1, 0, 70] <= 1
