"""Pins of the offloaded-decode oracle (CPU only), independent of its own replay:

* the hand-worked traces (``tests/golden/lru_hand_trace.txt``): per step, the fetched experts are
  the selected ones absent from the previous hand-listed state, the evicted ones are those of the
  previous state missing from the next, and the state after each step is the listed one (LRU,
  FIFO, LFU);
* set identities on random traces, checked from the trajectory alone: the fetched experts are
  exactly the selected ones not cached before the step; every selected expert is cached after
  it; nothing selected is evicted; the state after the step is the previous one minus the evicted
  plus the fetched; a full cache evicts one expert per fetch, a non-full one none;
* the layer output of a decode equals the plain layer on the same tokens, and the fetches per
  step equal K - hits (Eq. 5).
"""

import numpy as np
import pytest

from conftest import golden_path
from oracle import cache as C
from oracle import ffn as O
from oracle import offload as OF
from oracle import routing as R


def _hand():
    info, steps, section = {}, [], None
    with open(golden_path("lru_hand_trace.txt")) as fh:
        for line in fh:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            if line == "steps:":
                section = "steps"
                continue
            head = line.split()[0]
            if section == "steps" and head.isdigit():
                steps.append([int(v) for v in line.split()])
                continue
            section = None
            info[head] = line[len(head):].strip()
    return info, steps


@pytest.mark.parametrize("policy,key", [(C.LRU, "B4_state"), (C.FIFO, "FIFO_B4_state"), (C.LFU, "LFU_B4_state")])
def test_hand_trace_fetch_and_evict_sets(policy, key):
    info, steps = _hand()
    E = int(info["E"])
    states = [[int(v) for v in s.split(",")] for s in info[key].split("|")]
    traj = []
    C.replay_stream(steps, E, 4, policy, trajectory=traj)
    prev = []
    for t, A in enumerate(steps):
        assert traj[t]["cache"] == states[t]
        assert traj[t]["fetched"] == sorted(set(A) - set(prev))
        assert sorted(traj[t]["evicted"]) == sorted(set(prev) - set(states[t]))
        prev = states[t]


@pytest.mark.parametrize("policy", [C.LRU, C.LFU, C.FIFO])
@pytest.mark.parametrize("E,K,B", [(8, 2, 4), (16, 4, 6), (64, 6, 12), (8, 2, 2)])
def test_trajectory_set_identities(policy, E, K, B):
    g = np.random.default_rng(E * 100 + K * 10 + B + policy)
    steps = [sorted(g.choice(E, K, replace=False).tolist()) for _ in range(300)]
    traj = []
    f, h, final, _, bad = C.replay_stream(steps, E, B, policy, trajectory=traj)
    assert not bad and final == traj[-1]["cache"]
    prev = []
    for t, A in enumerate(steps):
        r = traj[t]
        cur = r["cache"]
        assert sorted(r["fetched"]) == sorted(set(A) - set(prev))
        assert set(A) <= set(cur) and len(cur) == len(set(cur)) <= B
        assert not set(r["evicted"]) & set(A)
        assert set(cur) == (set(prev) - set(r["evicted"])) | set(r["fetched"])
        assert len(r["evicted"]) == max(0, len(prev) + len(r["fetched"]) - B)
        assert f[t] == len(r["fetched"]) and f[t] + h[t] == K
        prev = cur


def test_decode_output_is_the_plain_layer_and_counts_follow_eq5():
    g = np.random.default_rng(3)
    N, d, F, E, K, S = 30, 16, 12, 8, 2, 1
    xs = g.standard_normal((N, d))
    wr = g.standard_normal((E, d)) * 0.5
    wgu = g.standard_normal((E, 2 * F, d)) / np.sqrt(d)
    wd = g.standard_normal((E, d, F)) / np.sqrt(F)
    sgu = g.standard_normal((S, 2 * F, d)) / np.sqrt(d)
    sd = g.standard_normal((S, d, F)) / np.sqrt(F)
    prior = np.array([0.3, 0.02, 0.3, 0.02, 0.02, 0.3, 0.02, 0.02])
    out = OF.decode_steps(xs, wr, wgu, wd, K, R.SOFT_PRIOR, R.GATE_RENORM, 4, C.LFU, prior=prior,
                          ws_gate_up=sgu, ws_down=sd)
    idx, gate, _ = R.route_logits(R.router_logits(xs, wr), K, R.SOFT_PRIOR, R.GATE_RENORM, prior=prior)
    np.testing.assert_array_equal(out["idx"], idx)
    np.testing.assert_array_equal(out["y"], O.moe_layer(xs, idx, gate, wgu, wd, sgu, sd))
    assert (out["f"] + out["h"] == K).all()
    assert out["f"].sum() == sum(len(x) for x in out["fetched"])
    assert OF.expert_bytes(4096, 14336) == 3 * 4096 * 14336 * 2
