"""GPU parity of maskmoe_offload_decode_step (batch-1 decode of one layer with the routed experts in
pinned host memory and a B-slot device pool) against the oracle's offloaded decode.

Per step, on inputs whose oracle routing has no near-tie (every margin > 2e-3, checked):
* the selected experts are the oracle's and the step fetches exactly the oracle's number of
  experts (bit-exact), and the cache state after the step (cached experts in recency or insertion
  order, LFU counts) equals the oracle's;
* y is within the layer's bf16 bound of the oracle, and bit-identical to maskmoe_layer_forward of
  the same token with every expert resident (same kernels, weights read from the pool);
* after the sequence, every pool slot that the state names holds its expert's weights bit for bit.
"""

import numpy as np
import pytest
import torch

import gpu_util as U
from oracle import cache as C
from oracle import offload as OF
from paper_2609_34077_amd import _lib as L
from paper_2609_34077_amd import synth

pytestmark = pytest.mark.gpu
MIN_MARGIN = 2e-3


def _pinned(a):
    return torch.from_numpy(np.ascontiguousarray(a)).view(torch.bfloat16).pin_memory()


def _decode(cfg, inp, B, policy, state=None, packed=False):
    """Runs the cfg.T tokens of inp one step at a time; returns per-step results. packed: the
    host copies (and the shared experts) in the packed layout, packed on the device."""
    E, K, d = cfg.E, cfg.K, cfg.d
    host_gu, host_dn = _pinned(inp["w_gate_up"]), _pinned(inp["w_down"])
    if packed:
        pg, pd = L.maskmoe_pack_expert_weights(U.dev(inp["w_gate_up"]), U.dev(inp["w_down"]))
        host_gu, host_dn = pg.cpu().pin_memory(), pd.cpu().pin_memory()
    slots_gu = torch.zeros((B, 2 * cfg.F, d), dtype=torch.bfloat16, device="cuda")
    slots_dn = torch.zeros((B, d, cfg.F), dtype=torch.bfloat16, device="cuda")
    st = L.offload_empty_state(E, B) if state is None else state
    xs = U.dev(inp["x"])
    wr = U.dev(inp["w_router"])
    sgu = U.dev(inp["ws_gate_up"]) if cfg.n_shared else None
    sdn = U.dev(inp["ws_down"]) if cfg.n_shared else None
    if packed and cfg.n_shared:
        sgu, sdn = L.maskmoe_pack_expert_weights(sgu, sdn)
    counters = torch.zeros(2, dtype=torch.int64, device="cuda")
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    mp = dict(prior=inp["prior"]) if cfg.route_mode == L.ROUTE_SOFT_PRIOR else dict(mask=inp["mask"])
    out = dict(y=[], idx=[], f=[], state=[], y_resident=[])
    for n in range(cfg.T):
        idx = torch.empty((1, K), dtype=torch.int32, device="cuda")
        gate = torch.empty((1, K), dtype=torch.float32, device="cuda")
        before = counters[0].item()
        y = L.maskmoe_offload_decode_step(xs[n:n + 1], wr, host_gu, host_dn, slots_gu, slots_dn, st, K,
                                          cfg.route_mode, cfg.gate_mode, policy, ws_gate_up=sgu, ws_down=sdn,
                                          counters=counters, dev_error=err, topk_idx=idx, topk_gate=gate,
                                          weight_layout=L.LAYOUT_PACKED if packed else L.LAYOUT_ROWS, **mp)
        torch.cuda.synchronize()
        out["f"].append(counters[0].item() - before)
        out["y"].append(y.clone())
        out["idx"].append(idx.cpu().numpy()[0])
        out["state"].append(st.cpu().numpy().copy())
    out["counters"] = counters.cpu().numpy()
    out["err"] = int(err.item())
    out["slots"] = (slots_gu, slots_dn)
    out["host"] = (host_gu, host_dn)
    out["xs"], out["wr"], out["sgu"], out["sdn"], out["mp"] = xs, wr, sgu, sdn, mp
    return out


def _check(cfg, B, policy, check_resident=True):
    U.say(f"offload {cfg.name} N={cfg.T} d={cfg.d} F={cfg.F} E={cfg.E} K={cfg.K} shared={cfg.n_shared} "
          f"B={B} policy={policy}")
    inp = synth.make_layer(cfg)
    w = lambda a: synth.widen(a, "bf16")
    mp = dict(prior=inp["prior"]) if cfg.route_mode == L.ROUTE_SOFT_PRIOR else dict(mask=inp["mask"])
    ref = OF.decode_steps(w(inp["x"]), w(inp["w_router"]), inp["w_gate_up"], inp["w_down"], cfg.K, cfg.route_mode,
                          cfg.gate_mode, B, policy, ws_gate_up=inp["ws_gate_up"] if cfg.n_shared else None,
                          ws_down=inp["ws_down"] if cfg.n_shared else None, widen=w, **mp)
    assert ref["margin"].min() > MIN_MARGIN, "inputs chosen without near-ties"
    got = _decode(cfg, inp, B, policy)
    E = cfg.E
    worst = 0.0
    for n in range(cfg.T):
        assert sorted(got["idx"][n]) == sorted(ref["idx"][n]), n
        assert got["f"][n] == ref["f"][n], (n, got["f"][n], ref["f"][n])
        order = got["state"][n][:B]
        want = ref["cache"][n] + [-1] * (B - len(ref["cache"][n]))
        assert order.tolist() == want, (n, order, want)
        slot_of = got["state"][n][B + E:]
        cached = set(ref["cache"][n])
        assert all((slot_of[e] >= 0) == (e in cached) for e in range(E))
        assert len({int(slot_of[e]) for e in cached}) == len(cached)
        worst = max(worst, U.normalized_max_error(U.y_to_f64(got["y"][n])[0:1], ref["y"][n:n + 1]))
    U.say(f"  fetches {int(got['counters'][0])} (oracle {int(ref['f'].sum())}), hits {int(got['counters'][1])}, "
          f"max normalised error {worst:.2e}")
    assert worst <= U.BF16_TOL
    assert int(got["counters"][0]) == int(ref["f"].sum()) and int(got["counters"][1]) == int(ref["h"].sum())
    assert got["err"] == 0
    if policy == C.LFU:
        assert got["state"][-1][B:B + E].tolist() == list(ref["final_counts"])
    # every slot the state names holds its expert's weights
    st = got["state"][-1]
    slots_gu, slots_dn = got["slots"]
    host_gu, host_dn = got["host"]
    for e in ref["final_state"]:
        s = int(st[B + E + e])
        assert torch.equal(slots_gu[s].cpu(), host_gu[e]) and torch.equal(slots_dn[s].cpu(), host_dn[e]), e
    if check_resident:   # the same kernels with every expert resident give the same bits
        wgu, wdn = U.dev(inp["w_gate_up"]), U.dev(inp["w_down"])
        for n in range(cfg.T):
            y0 = L.maskmoe_layer_forward(got["xs"][n:n + 1], got["wr"], wgu, wdn, cfg.K, cfg.route_mode,
                                         cfg.gate_mode, ws_gate_up=got["sgu"], ws_down=got["sdn"], **got["mp"])
            torch.cuda.synchronize()
            assert torch.equal(y0, got["y"][n]), n
    return got, ref


SMALL = synth.LayerConfig("offload_small", T=48, d=256, F=512, E=8, K=2, route_mode=L.ROUTE_SOFT_PRIOR,
                          mask_set=(0, 2, 5, 7), delta=0.2, seed=87)
SHARED = synth.LayerConfig("offload_shared", T=40, d=256, F=128, E=16, K=4, n_shared=1,
                           route_mode=L.ROUTE_SOFT_PRIOR, gate_mode=L.GATE_P, mask_set=tuple(range(0, 16, 2)),
                           delta=1.0, seed=87)


@pytest.mark.parametrize("policy", [C.LRU, C.LFU, C.FIFO], ids=["lru", "lfu", "fifo"])
def test_offload_small(policy):
    _check(SMALL, 4, policy)


@pytest.mark.parametrize("policy", [C.LRU, C.LFU, C.FIFO], ids=["lru", "lfu", "fifo"])
def test_offload_shared_experts(policy):
    _check(SHARED, 6, policy)


def test_offload_cache_of_every_expert_fetches_each_once():
    """B = E: only first uses fetch (the number of distinct experts)."""
    got, ref = _check(SMALL.with_(name="offload_b_e", T=24), 8, C.LRU, check_resident=False)
    assert int(got["counters"][0]) == len(np.unique(np.concatenate(got["idx"])))


def test_offload_inconsistent_state_is_reset_and_reported():
    cfg = SMALL.with_(name="offload_bad_state", T=1)
    inp = synth.make_layer(cfg)
    B, E = 4, cfg.E
    st = L.offload_empty_state(E, B)
    st[0], st[1] = 3, 3                      # an expert listed twice
    got = _decode(cfg, inp, B, C.LRU, state=st)
    assert got["err"] == 1
    assert got["f"][0] == cfg.K               # started from an empty cache
    s = got["state"][0]
    assert sorted(s[:B][s[:B] >= 0].tolist()) == sorted(got["idx"][0].tolist())
    st2 = L.offload_empty_state(E, B)
    st2[0], st2[B + E + 0] = 0, 7            # slot out of range for a cached expert
    got2 = _decode(cfg, inp, B, C.LRU, state=st2)
    assert got2["err"] == 1 and got2["f"][0] == cfg.K


def test_offload_mixtral_full_size():
    """Mixtral-shaped layer (d = 4096, F = 14336, 8 experts of 352 MB in pinned host memory), 8 steps, B = 4."""
    cfg = synth.mixtral_decode_config(8).with_(name="offload_mixtral", delta=0.2, seed=2)
    _check(cfg, 4, C.LRU)


@pytest.mark.parametrize("cfg", [SMALL, SHARED], ids=lambda c: c.name)
def test_offload_packed_weights_match_row_major_bitwise(cfg):
    """Packed host copies (and shared experts): the same selections, fetches, cache states and
    output bits as the row-major offloaded decode."""
    U.say(f"offload packed vs row-major {cfg.name}")
    inp = synth.make_layer(cfg)
    a = _decode(cfg, inp, 4, C.LFU)
    b = _decode(cfg, inp, 4, C.LFU, packed=True)
    assert a["f"] == b["f"] and a["err"] == b["err"] == 0
    for n in range(cfg.T):
        assert np.array_equal(a["idx"][n], b["idx"][n]) and np.array_equal(a["state"][n], b["state"][n]), n
        assert torch.equal(a["y"][n].view(torch.int16), b["y"][n].view(torch.int16)), n
