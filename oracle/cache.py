"""Oracle: per-layer expert cache of the trace simulator (pure Python). Test infrastructure only.

Section 4.1 (Simulation): each layer keeps a cache of B routed experts
(K <= B < E; B >= E is accepted and then never evicts). Caches start empty
unless a state is given, initial fills count as misses, every miss is one
fetch and a full cache evicts one entry per miss under the LRU, LFU or FIFO
policy (Section 4.1; Table 2). Shared experts are not part of the trace.
Eq. 5: h_{l,t} counts the selected experts already cached,
f_{l,t} = K - h_{l,t} counts the misses, HR = sum h / (N L K) and
Fetches/tok = sum f / N, so Fetches/tok = L K (1 - HR).

Readings of what the paper leaves open:
* within one step the hits are handled first, in ascending expert index,
  then the misses are inserted in ascending expert index; a miss evicts one
  cached expert that is not selected at this step;
* LRU evicts the least recently used such expert;
* FIFO evicts the one inserted earliest (hits do not refresh it);
* LFU evicts the one accessed least often, counting every access of the
  stream so far (counts survive eviction), ties going to the least recently
  used;
* a trace entry outside [0, E) or repeating an earlier entry of the same
  step is skipped (it counts neither as hit nor as miss) and reported;
* a cache state lists the cached experts from least to most recently used
  (LRU, LFU) or from first to last inserted (FIFO); LFU's access counts are
  kept per expert next to it.
"""

from __future__ import annotations

from typing import Iterable, List, Optional, Sequence, Tuple

import numpy as np

LRU, LFU, FIFO = 0, 1, 2
POLICIES = {"LRU": LRU, "LFU": LFU, "FIFO": FIFO}


def step_set(entries: Iterable[int], E: int) -> Tuple[List[int], bool]:
    """Distinct in-range experts of one step, ascending; and whether any entry was skipped."""
    seen: List[int] = []
    bad = False
    for e in entries:
        e = int(e)
        if e < 0 or e >= E or e in seen:
            bad = True
            continue
        seen.append(e)
    return sorted(seen), bad


def replay_stream(steps: Sequence[Sequence[int]], E: int, B: int, policy: int = LRU,
                  state: Optional[Sequence[int]] = None, counts: Optional[Sequence[int]] = None,
                  trajectory: Optional[list] = None):
    """Replay one (layer, stream) trace through a B-slot cache under ``policy``.

    ``cache`` is kept as an ordered list: by last use (LRU, LFU) or by
    insertion (FIFO), oldest first. Returns ``(f, h, final_state,
    final_counts, bad)``. When ``trajectory`` is a list, one record per step
    is appended to it: ``fetched`` (the misses, in insertion order),
    ``evicted`` (in eviction order) and ``cache`` (the state after the step).
    """
    cache: List[int] = []
    for e in (state or []):
        e = int(e)
        if 0 <= e < E and e not in cache:
            cache.append(e)
    freq = [int(c) for c in counts] if counts is not None else [0] * E
    f: List[int] = []
    h: List[int] = []
    bad_any = False
    for entries in steps:
        A, bad = step_set(entries, E)
        bad_any |= bad
        for e in A:
            freq[e] += 1
        hits = [e for e in A if e in cache]
        misses = [e for e in A if e not in cache]
        if policy in (LRU, LFU):
            for e in hits:                      # becomes most recently used
                cache.remove(e)
                cache.append(e)
        evicted: List[int] = []
        for e in misses:
            if len(cache) >= B:
                candidates = [c for c in cache if c not in A]   # oldest first
                if policy == LFU:
                    low = min(freq[c] for c in candidates)
                    victim = next(c for c in candidates if freq[c] == low)
                else:
                    victim = candidates[0]
                cache.remove(victim)
                evicted.append(victim)
            cache.append(e)
        h.append(len(hits))
        f.append(len(misses))
        if trajectory is not None:
            trajectory.append(dict(fetched=list(misses), evicted=evicted, cache=list(cache)))
    return f, h, cache, freq, bad_any


def lru_stream(steps: Sequence[Sequence[int]], E: int, B: int,
               state: Optional[Sequence[int]] = None):
    """LRU replay of one stream: ``(f, h, final_state, bad)``."""
    f, h, cache, _, bad = replay_stream(steps, E, B, LRU, state)
    return f, h, cache, bad


def cache_fetches(trace: np.ndarray, E: int, B: int, state: Optional[np.ndarray] = None,
                  policy: int = LRU, counts: Optional[np.ndarray] = None):
    """Replay a trace [L,S,N,K] with one independent cache per (layer, stream).

    ``state`` is an optional ``[L,S,B]`` int array of initial caches (-1 =
    empty slot) and ``counts`` optional ``[L,S,E]`` LFU access counts.
    Returns ``fetches [L,S]``, ``hits [L,S]`` (int64), ``f_per_step
    [L,S,N]`` (uint8), the final state ``[L,S,B]`` and whether any trace
    entry was skipped; with ``policy == LFU`` the final counts ``[L,S,E]``
    are appended.
    """
    trace = np.asarray(trace)
    L, S, N, K = trace.shape
    fetches = np.zeros((L, S), dtype=np.int64)
    hits = np.zeros((L, S), dtype=np.int64)
    fps = np.zeros((L, S, N), dtype=np.uint8)
    final = np.full((L, S, B), -1, dtype=np.int32)
    fcounts = np.zeros((L, S, E), dtype=np.int32)
    bad_any = False
    for l in range(L):
        for s in range(S):
            init = None if state is None else [int(e) for e in state[l, s] if e >= 0]
            c0 = None if counts is None else counts[l, s].tolist()
            f, h, c, fr, bad = replay_stream(trace[l, s].tolist(), E, B, policy, init, c0)
            fetches[l, s] = sum(f)
            hits[l, s] = sum(h)
            fps[l, s] = f
            final[l, s, :len(c)] = c
            fcounts[l, s] = fr
            bad_any |= bad
    if policy == LFU:
        return fetches, hits, fps, final, bad_any, fcounts
    return fetches, hits, fps, final, bad_any


def hit_rate(total_hits: int, N: int, L: int, K: int) -> float:
    """HR = (1 / (N L K)) * sum_l sum_t h_{l,t}  (Eq. 5)."""
    return total_hits / (N * L * K)


def fetches_per_token(total_fetches: int, N: int) -> float:
    """Fetches/tok = (1 / N) * sum_l sum_t f_{l,t}  (Eq. 5): summed over layers, averaged over steps."""
    return total_fetches / N
