"""Seeded synthetic inputs for the masked MoE layer and the routing/fetch trace.

This module holds no arithmetic of the method. It only draws random numbers,
scales them to the stated standard deviations, rounds them to the storage
type, runs the AR(1) hidden-state recursion of the trace workload and builds
the mask and prior arrays that the layer takes as inputs. The CPU oracle and
the HIP path both consume what it returns; neither is imported here.

Workload shapes follow the models of the paper (Mixtral-8x7B: d=4096,
F=14336, E=8, K=2, 32 MoE layers; DeepSeek-V2-Lite: d=2048, F=1408, E=64
routed + 2 shared experts, K=6; Appendix A, Table 4) and its cache budgets
(4 experts per layer for Mixtral, 12 for DeepSeek; Section 4.1, Simulation).
The paper's data (OpenHermes, ShareGPT) and trained weights are not
available: every input here is a seeded stand-in of the same shape.

Storage conventions
-------------------
* bf16 tensors are returned as ``uint16`` arrays holding the bf16 bit
  pattern, rounded from float32 with round-to-nearest-even.
* f32 tensors are returned as ``float32`` arrays.
* ``widen(a, dtype)`` returns the exact float64 values of either form.
* Expert weights: ``w_gate_up`` is ``[E, 2F, d]`` (rows ``0..F-1`` are the
  gate projection, rows ``F..2F-1`` the up projection), ``w_down`` is
  ``[E, d, F]``; shared experts use the same layout with ``n_shared`` in
  place of ``E``.
"""

from __future__ import annotations

import concurrent.futures as _cf
import dataclasses
import os
from typing import Dict, List, Optional, Sequence

import numpy as np

ROUTE_PLAIN, ROUTE_HARD_MASK, ROUTE_SOFT_PRIOR = 0, 1, 2
GATE_P, GATE_RENORM = 0, 1


# ---------------------------------------------------------------- storage

def bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (round-to-nearest-even); return the bits."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact float32 value of bf16 bit patterns."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def widen(a: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float64 values of a stored tensor (bf16 bits or float32)."""
    if dtype == "bf16":
        return bf16_to_f32(a).astype(np.float64)
    return np.asarray(a, dtype=np.float64)


def _store(a: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return bf16_bits(a)
    return np.ascontiguousarray(a, dtype=np.float32)


def _normal(seq: np.random.SeedSequence, shape, std: float, dtype: str) -> np.ndarray:
    g = np.random.Generator(np.random.PCG64(seq))
    a = g.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        a *= np.float32(std)
    return _store(a, dtype)


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


# ---------------------------------------------------------------- configs

@dataclasses.dataclass(frozen=True)
class LayerConfig:
    """One masked MoE layer workload."""

    name: str
    T: int                      # tokens
    d: int                      # hidden size
    F: int                      # expert FFN width
    E: int                      # routed experts
    K: int                      # experts per token
    n_shared: int = 0           # always-on shared experts
    dtype: str = "bf16"         # "bf16" or "f32"
    route_mode: int = ROUTE_SOFT_PRIOR
    gate_mode: int = GATE_RENORM
    mask_set: Optional[Sequence[int]] = None   # experts kept by the mask / favoured by the prior
    delta: float = 1.0          # prior strength: mask logit of the kept experts
    seed: int = 0

    def with_(self, **kw) -> "LayerConfig":
        return dataclasses.replace(self, **kw)


def tiny_config(route_mode: int = ROUTE_HARD_MASK) -> LayerConfig:
    """Tiny fp32 layer: d=256, F=512, E=8, top-2 renormalised, mask {0,2,5,7}, 64 tokens."""
    return LayerConfig("tiny_f32", T=64, d=256, F=512, E=8, K=2, dtype="f32",
                       route_mode=route_mode, gate_mode=GATE_RENORM, mask_set=(0, 2, 5, 7))


def mixtral_decode_config(T: int) -> LayerConfig:
    """Mixtral-shaped decode layer, soft prior from a 4-expert mask, T in {1, 4, 16}."""
    return LayerConfig(f"mixtral_decode_t{T}", T=T, d=4096, F=14336, E=8, K=2,
                       route_mode=ROUTE_SOFT_PRIOR, gate_mode=GATE_RENORM, mask_set=(0, 2, 5, 7))


def mixtral_ft_config(T: int = 8192) -> LayerConfig:
    """Mixtral-shaped fine-tuning forward: hard mask keeping 4 experts, 8192 tokens (4 x 2048)."""
    return LayerConfig(f"mixtral_ft_t{T}", T=T, d=4096, F=14336, E=8, K=2,
                       route_mode=ROUTE_HARD_MASK, gate_mode=GATE_RENORM, mask_set=(0, 2, 5, 7))


def deepseek_mask_set(E: int = 64, size: int = 12, seed: int = 0) -> List[int]:
    """The 12-expert set of the DeepSeek-shaped layer: a seeded draw without replacement."""
    g = np.random.default_rng(seed)
    return sorted(int(i) for i in g.choice(E, size, replace=False))


def deepseek_config(route_mode: int = ROUTE_SOFT_PRIOR, T: int = 4096) -> LayerConfig:
    """DeepSeek-V2-Lite-shaped layer: d=2048, 64 routed + 2 shared experts of width 1408, top-6, g=p."""
    return LayerConfig(f"deepseek_t{T}_{'hard' if route_mode == ROUTE_HARD_MASK else 'soft'}",
                       T=T, d=2048, F=1408, E=64, K=6, n_shared=2,
                       route_mode=route_mode, gate_mode=GATE_P,
                       mask_set=tuple(deepseek_mask_set()))


# ---------------------------------------------------------------- mask / prior inputs

def binary_mask(E: int, keep: Sequence[int]) -> np.ndarray:
    """Binary expert mask m in {0,1}^E with ones at ``keep`` (uint8)."""
    m = np.zeros(E, dtype=np.uint8)
    m[list(keep)] = 1
    return m


def concentrated_prior(E: int, keep: Optional[Sequence[int]], delta: float) -> np.ndarray:
    """A strictly positive prior over E experts that favours ``keep``.

    The synthetic stand-in for a learned prior: the mask logits are
    ``delta`` on the kept experts and 0 elsewhere, and the prior is their
    normalised exponentials (float32). ``keep=None`` or ``delta=0`` gives
    the uniform prior ("zero prior").
    """
    logits = np.zeros(E, dtype=np.float64)
    if keep is not None:
        logits[list(keep)] = delta
    w = np.exp(logits - logits.max())
    return (w / w.sum()).astype(np.float32)


# ---------------------------------------------------------------- layer inputs

def make_layer(cfg: LayerConfig, with_x: bool = True, threads: Optional[int] = None) -> Dict[str, np.ndarray]:
    """Seeded inputs of one layer.

    Independent random streams (``SeedSequence(cfg.seed).spawn``) are used for
    the router, each expert's gate/up and down projections, the shared experts
    and the tokens, so any tensor can be regenerated alone and the result does
    not depend on the number of threads.

    Returns ``x [T,d]``, ``w_router [E,d]``, ``w_gate_up [E,2F,d]``,
    ``w_down [E,d,F]``, ``ws_gate_up [n_shared,2F,d]``, ``ws_down
    [n_shared,d,F]`` (empty when ``n_shared == 0``), ``mask uint8 [E]`` and
    ``prior float32 [E]``.
    """
    E, F, d, ns, dt = cfg.E, cfg.F, cfg.d, cfg.n_shared, cfg.dtype
    root = np.random.SeedSequence(cfg.seed)
    s_router, s_experts, s_shared, s_x = root.spawn(4)
    exp_seqs = s_experts.spawn(E)
    sh_seqs = s_shared.spawn(max(ns, 1))

    out: Dict[str, np.ndarray] = {}
    out["w_router"] = _normal(s_router, (E, d), 0.02, dt)
    elem = np.uint16 if dt == "bf16" else np.float32
    w_gu = np.empty((E, 2 * F, d), dtype=elem)
    w_dn = np.empty((E, d, F), dtype=elem)
    ws_gu = np.empty((ns, 2 * F, d), dtype=elem)
    ws_dn = np.empty((ns, d, F), dtype=elem)

    def fill(dst_gu, dst_dn, i, seq):
        a, b = seq.spawn(2)
        dst_gu[i] = _normal(a, (2 * F, d), 1.0 / np.sqrt(d), dt)
        dst_dn[i] = _normal(b, (d, F), 1.0 / np.sqrt(F), dt)

    jobs = [(w_gu, w_dn, i, exp_seqs[i]) for i in range(E)]
    jobs += [(ws_gu, ws_dn, i, sh_seqs[i]) for i in range(ns)]
    with _cf.ThreadPoolExecutor(max_workers=threads or _threads()) as pool:
        list(pool.map(lambda j: fill(*j), jobs))
    out["w_gate_up"], out["w_down"] = w_gu, w_dn
    out["ws_gate_up"], out["ws_down"] = ws_gu, ws_dn
    if with_x:
        out["x"] = _normal(s_x, (cfg.T, d), 1.0, dt)
    out["mask"] = binary_mask(E, cfg.mask_set if cfg.mask_set is not None else range(E))
    out["prior"] = concentrated_prior(E, cfg.mask_set, cfg.delta)
    return out


def make_lora(cfg: LayerConfig, rank: int = 8, alpha: float = 16.0, b_std: float = 0.05) -> Dict[str, object]:
    """Seeded low-rank adapters of every expert (rank 8, alpha 16 by default, as in the paper's
    Stage-2 set-up). A ~ N(0, 1/in) (the scale of the usual uniform initialisation); B, zero at
    initialisation, stands in for a trained adapter with std ``b_std`` (0.05 gives an adapter
    term of about a quarter of W x for unit-variance tokens).

    Returns rank, alpha and, in the storage type of ``cfg.dtype``: ``a_gate_up [E,2r,d]`` (the
    gate adapter's A rows, then the up adapter's), ``b_gate_up [E,2F,r]``, ``a_down [E,r,F]``,
    ``b_down [E,d,r]`` and ``as_*`` / ``bs_*`` for the ``n_shared`` shared experts.
    """
    E, F, d, ns, dt = cfg.E, cfg.F, cfg.d, cfg.n_shared, cfg.dtype
    seqs = np.random.SeedSequence([cfg.seed, 104729, rank]).spawn(8)
    out: Dict[str, object] = dict(rank=rank, alpha=alpha)
    out["a_gate_up"] = _normal(seqs[0], (E, 2 * rank, d), 1.0 / np.sqrt(d), dt)
    out["b_gate_up"] = _normal(seqs[1], (E, 2 * F, rank), b_std, dt)
    out["a_down"] = _normal(seqs[2], (E, rank, F), 1.0 / np.sqrt(F), dt)
    out["b_down"] = _normal(seqs[3], (E, d, rank), b_std, dt)
    out["as_gate_up"] = _normal(seqs[4], (ns, 2 * rank, d), 1.0 / np.sqrt(d), dt)
    out["bs_gate_up"] = _normal(seqs[5], (ns, 2 * F, rank), b_std, dt)
    out["as_down"] = _normal(seqs[6], (ns, rank, F), 1.0 / np.sqrt(F), dt)
    out["bs_down"] = _normal(seqs[7], (ns, d, rank), b_std, dt)
    return out


def layer_tokens(cfg: LayerConfig) -> np.ndarray:
    """The tokens ``x [T,d]`` that ``make_layer(cfg)`` returns, drawn alone (same stream)."""
    s_x = np.random.SeedSequence(cfg.seed).spawn(4)[3]
    return _normal(s_x, (cfg.T, cfg.d), 1.0, cfg.dtype)


def make_tokens(cfg: LayerConfig, T: int, stream: int) -> np.ndarray:
    """Extra token batches x ~ N(0,1) [T,d] from a stream keyed by ``stream`` (>= 1)."""
    seq = np.random.SeedSequence([cfg.seed, 7919, stream])
    return _normal(seq, (T, cfg.d), 1.0, cfg.dtype)


# ---------------------------------------------------------------- routing / fetch trace

@dataclasses.dataclass(frozen=True)
class TraceConfig:
    """Routing-and-fetch trace: L independent Mixtral-shaped routers over AR(1) streams."""

    L: int = 32
    E: int = 8
    K: int = 2
    d: int = 4096
    S: int = 256        # sequences (independent cache streams)
    N: int = 512        # decode steps per sequence
    B: int = 4          # cache slots per layer
    rho: float = 0.9    # AR(1) coefficient
    delta: float = 1.0  # prior strength on each layer's 4-expert set
    set_size: int = 4
    seed: int = 0


def trace_layer_sets(cfg: TraceConfig) -> List[List[int]]:
    """Per-layer random ``set_size``-expert sets, drawn without replacement."""
    g = np.random.default_rng(np.random.SeedSequence([cfg.seed, 101]))
    return [sorted(int(i) for i in g.choice(cfg.E, cfg.set_size, replace=False)) for _ in range(cfg.L)]


def make_trace_inputs(cfg: TraceConfig, threads: Optional[int] = None) -> Dict[str, np.ndarray]:
    """Inputs of the routing-and-fetch trace.

    ``x`` is ``[S*N, d]`` bf16 bits in sequence-major token order
    (``t = s*N + n``), following ``x_0 ~ N(0,I)``,
    ``x_n = rho*x_{n-1} + sqrt(1-rho^2)*eps_n`` with the recursion carried in
    float64 and each step stored as bf16. The same hidden states feed every
    layer. ``w_router`` is ``[L,E,d]`` (std 0.02), ``prior`` is ``[L,E]``
    (each layer favours its own set) and ``prior_zero`` the uniform prior.
    """
    L, E, d, S, N = cfg.L, cfg.E, cfg.d, cfg.S, cfg.N
    root = np.random.SeedSequence(cfg.seed)
    s_router, s_x = root.spawn(2)
    out: Dict[str, np.ndarray] = {}
    out["w_router"] = _normal(s_router, (L, E, d), 0.02, "bf16")
    x = np.empty((S, N, d), dtype=np.uint16)
    seqs = s_x.spawn(S)
    c = np.sqrt(1.0 - cfg.rho * cfg.rho)

    def one(s):
        g = np.random.Generator(np.random.PCG64(seqs[s]))
        h = g.standard_normal(d)
        x[s, 0] = bf16_bits(h.astype(np.float32))
        for n in range(1, N):
            h = cfg.rho * h + c * g.standard_normal(d)
            x[s, n] = bf16_bits(h.astype(np.float32))

    with _cf.ThreadPoolExecutor(max_workers=threads or _threads()) as pool:
        list(pool.map(one, range(S)))
    out["x"] = x.reshape(S * N, d)
    sets = trace_layer_sets(cfg)
    out["sets"] = np.array(sets, dtype=np.int32)
    out["prior"] = np.stack([concentrated_prior(E, s, cfg.delta) for s in sets])
    out["prior_zero"] = np.stack([concentrated_prior(E, None, 0.0) for _ in sets])
    return out


def random_trace(L: int, S: int, N: int, K: int, E: int, seed: int = 0, locality: float = 0.0) -> np.ndarray:
    """A random expert-selection trace ``[L,S,N,K]`` (int32), K distinct experts per step.

    With probability ``locality`` a step keeps each expert of the previous
    step (then refills to K distinct experts at random), which gives traces
    with cache reuse.
    """
    g = np.random.default_rng(seed)
    tr = np.empty((L, S, N, K), dtype=np.int32)
    for l in range(L):
        for s in range(S):
            prev: List[int] = []
            for n in range(N):
                cur = [e for e in prev if g.random() < locality]
                while len(cur) < K:
                    e = int(g.integers(E))
                    if e not in cur:
                        cur.append(e)
                g.shuffle(cur)
                tr[l, s, n] = cur
                prev = cur
    return tr
