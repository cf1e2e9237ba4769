"""C-ABI checks that need no GPU: the library loads, exports every declared entry point,
and rejects invalid arguments before touching the device; workspace sizing is monotone."""

import ctypes
import os
import re

import numpy as np
import pytest

from conftest import ROOT
from paper_2609_34077_amd import _lib as L

HEADER = os.path.join(ROOT, "include", "maskmoe.h")

pytestmark = pytest.mark.skipif(not os.path.exists(L.LIB_PATH), reason="libmaskmoe.so not built")

FAKE = 0x10000  # a 256-byte aligned non-null address; only used where validation must fail


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:int|size_t|const char\*)\s+(maskmoe_\w+)\s*\(", text, re.M)))


def test_library_exports_every_declared_function():
    names = declared_functions()
    assert set(names) == set(L.EXPORTS)
    lib = ctypes.CDLL(L.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings():
    lib = L.load()
    for code in range(6):
        assert lib.maskmoe_status_string(code)
    assert lib.maskmoe_status_string(99) == b"unknown status"


def _route(desc, Lyr=1, x=FAKE, w=FAKE, mask=None, prior=None, idx=FAKE, gate=FAKE, margin=None, ws=None,
           ws_bytes=0):
    lib = L.load()
    return lib.maskmoe_route(ctypes.byref(desc), Lyr, x, w, mask, prior, idx, gate, margin, ws, ws_bytes, None)


def test_route_workspace_bytes():
    """Split routing (bf16, T >= 512, E <= 64) asks for fp32 [L, T, E] router logits; else none."""
    lib = L.load()
    nb = lambda Lyr=1, **k: lib.maskmoe_route_workspace_bytes(
        ctypes.byref(L.make_desc(**{**dict(T=1024, d=64, E=8, K=2, dtype=L.BF16), **k})), Lyr)
    assert nb() == 1024 * 8 * 4
    assert nb(Lyr=32) == 32 * 1024 * 8 * 4
    assert nb(E=64, K=6) == 1024 * 64 * 4
    assert nb(T=511) == 0 and nb(E=65) == 0 and nb(dtype=L.F32) == 0
    assert nb(Lyr=0) == 0 and nb(K=0) == 0
    desc = L.make_desc(T=1024, d=64, E=8, K=2, dtype=L.BF16)
    assert _route(desc, ws=FAKE, ws_bytes=1024 * 8 * 4 - 1) == L.E_INVAL      # too small
    assert _route(desc, ws=FAKE + 8, ws_bytes=1 << 20) == L.E_INVAL          # misaligned


def test_route_rejects_invalid_arguments():
    good = dict(T=4, d=64, E=8, K=2, dtype=L.BF16, route_mode=L.ROUTE_PLAIN, gate_mode=L.GATE_RENORM)
    bad = [dict(T=-1), dict(d=0), dict(E=0), dict(E=257), dict(K=0), dict(K=9), dict(E=32, K=17),
           dict(dtype=7), dict(route_mode=3), dict(gate_mode=2)]
    for b in bad:
        desc = L.make_desc(**{**good, **b})
        assert _route(desc) == L.E_INVAL, b
    desc = L.make_desc(**good)
    assert _route(desc, Lyr=0) == L.E_INVAL
    assert _route(desc, x=None) == L.E_INVAL
    assert _route(desc, idx=None) == L.E_INVAL
    assert _route(desc, x=FAKE + 2) == L.E_INVAL          # misaligned
    assert _route(L.make_desc(**{**good, "d": 48})) == L.E_UNSUPPORTED


def test_route_rejects_bad_mask_and_prior():
    E, K = 8, 2
    hard = L.make_desc(T=4, d=64, E=E, K=K, route_mode=L.ROUTE_HARD_MASK)
    m = np.array([1, 0, 0, 0, 0, 0, 0, 0], np.uint8)                  # one expert < K
    assert _route(hard, mask=m.ctypes.data_as(ctypes.c_void_p)) == L.E_INVAL
    assert _route(hard, mask=None) == L.E_INVAL
    m2 = np.array([[1, 1, 0, 0, 0, 0, 0, 0], [0, 0, 0, 0, 0, 0, 0, 1]], np.uint8)   # second layer bad
    assert _route(hard, Lyr=2, mask=m2.ctypes.data_as(ctypes.c_void_p)) == L.E_INVAL
    soft = L.make_desc(T=4, d=64, E=E, K=K, route_mode=L.ROUTE_SOFT_PRIOR)
    for badv in (0.0, -0.1, np.inf, np.nan):
        p = np.full(E, 1.0 / E, np.float32)
        p[3] = badv
        assert _route(soft, prior=p.ctypes.data_as(ctypes.c_void_p)) == L.E_INVAL
    assert _route(soft, prior=None) == L.E_INVAL


def test_route_with_no_tokens_is_a_no_op():
    desc = L.make_desc(T=0, d=64, E=8, K=2)
    assert _route(desc, x=None, w=None, idx=None, gate=None) == L.OK


def _fwd(desc, ws_bytes=None, **kw):
    lib = L.load()
    a = dict(x=FAKE, w=FAKE, mask=None, prior=None, wgu=FAKE, wdn=FAKE, sgu=None, sdn=None, y=FAKE,
             idx=None, gate=None, ws=FAKE)
    a.update(kw)
    if ws_bytes is None:
        ws_bytes = lib.maskmoe_layer_workspace_bytes(ctypes.byref(desc))
    return lib.maskmoe_layer_forward(ctypes.byref(desc), a["x"], a["w"], a["mask"], a["prior"], a["wgu"],
                                     a["wdn"], a["sgu"], a["sdn"], a["y"], a["idx"], a["gate"], a["ws"],
                                     ws_bytes, None)


def test_layer_forward_rejects_invalid_arguments():
    lib = L.load()
    good = dict(T=32, d=128, E=8, K=2, F=256, n_shared=0, dtype=L.BF16, route_mode=L.ROUTE_PLAIN,
                gate_mode=L.GATE_RENORM)
    for b in (dict(F=0), dict(n_shared=-1), dict(n_shared=9), dict(K=0)):
        assert _fwd(L.make_desc(**{**good, **b}), ws_bytes=1 << 30) == L.E_INVAL, b
    desc = L.make_desc(**good)
    assert _fwd(desc, y=None) == L.E_INVAL
    assert _fwd(desc, wgu=None) == L.E_INVAL
    assert _fwd(desc, x=FAKE + 8) == L.E_INVAL
    assert _fwd(L.make_desc(**{**good, "n_shared": 1})) == L.E_INVAL       # shared weights missing
    need = lib.maskmoe_layer_workspace_bytes(ctypes.byref(desc))
    assert _fwd(desc, ws_bytes=need - 1) == L.E_WORKSPACE
    assert _fwd(desc, ws=None) == L.E_WORKSPACE
    assert _fwd(desc, ws=FAKE + 64) == L.E_WORKSPACE                        # not 256-byte aligned
    assert _fwd(L.make_desc(**{**good, "F": 96}), ws_bytes=1 << 30) == L.E_UNSUPPORTED
    assert _fwd(L.make_desc(**{**good, "d": 96}), ws_bytes=1 << 30) == L.E_UNSUPPORTED


def test_profiled_forward_needs_an_event_array():
    lib = L.load()
    desc = L.make_desc(T=32, d=128, E=8, K=2, F=256)
    ws = lib.maskmoe_layer_workspace_bytes(ctypes.byref(desc))
    assert lib.maskmoe_layer_forward_profiled(ctypes.byref(desc), FAKE, FAKE, None, None, FAKE, FAKE, None, None,
                                              FAKE, None, None, FAKE, ws, None, None) == L.E_INVAL


def test_noalloc_forward_checks_its_limit_before_touching_the_device():
    """The no-allocation entry point rejects a layer whose workspace exceeds its fixed scratch
    array (E_WORKSPACE) and an invalid desc (E_INVAL) before any HIP call."""
    lib = L.load()
    call = lambda desc: lib.maskmoe_layer_forward_noalloc(ctypes.byref(desc), FAKE, FAKE, None, None, FAKE, FAKE,
                                                          None, None, FAKE, None, None, None)
    big = L.make_desc(T=8192, d=4096, E=8, K=2, F=14336, dtype=L.BF16, route_mode=L.ROUTE_PLAIN)
    assert lib.maskmoe_layer_workspace_bytes(ctypes.byref(big)) > L.NOALLOC_SCRATCH_BYTES
    assert call(big) == L.E_WORKSPACE
    assert call(L.make_desc(T=16, d=4096, E=8, K=0, F=14336)) == L.E_INVAL
    # the decode batches of the Mixtral-shaped layer fit the array
    for T in (1, 4, 16):
        dec = L.make_desc(T=T, d=4096, E=8, K=2, F=14336, dtype=L.BF16, route_mode=L.ROUTE_SOFT_PRIOR,
                          weight_layout=L.LAYOUT_PACKED)
        assert lib.maskmoe_layer_workspace_bytes(ctypes.byref(dec)) <= L.NOALLOC_SCRATCH_BYTES


def _lora_fwd(desc, lora, ws_bytes=1 << 40, **kw):
    lib = L.load()
    a = dict(x=FAKE, w=FAKE, wgu=FAKE, wdn=FAKE, sgu=None, sdn=None, y=FAKE, ws=FAKE)
    a.update(kw)
    lp = ctypes.byref(lora) if lora is not None else None
    return lib.maskmoe_layer_forward_lora(ctypes.byref(desc), a["x"], a["w"], None, None, a["wgu"], a["wdn"],
                                          a["sgu"], a["sdn"], lp, a["y"], None, None, a["ws"], ws_bytes, None)


def test_lora_forward_rejects_invalid_arguments():
    lib = L.load()
    good = dict(T=32, d=128, E=8, K=2, F=256, n_shared=0, dtype=L.BF16, route_mode=L.ROUTE_PLAIN,
                gate_mode=L.GATE_RENORM)
    desc = L.make_desc(**good)

    def lora(rank=8, alpha=16.0, **ptrs):
        p = dict(a_gate_up=FAKE, b_gate_up=FAKE, a_down=FAKE, b_down=FAKE)
        p.update(ptrs)
        return L.Lora(rank, alpha, *[p.get(k) for k in L.LORA_KEYS])

    assert _lora_fwd(desc, None) == L.E_INVAL
    for bad in (dict(rank=0), dict(rank=17), dict(alpha=float("inf")), dict(alpha=float("nan")),
                dict(a_down=None), dict(b_gate_up=None), dict(a_gate_up=FAKE + 8)):
        assert _lora_fwd(desc, lora(**bad)) == L.E_INVAL, bad
    # shared experts need their adapters too
    sh = L.make_desc(**{**good, "n_shared": 1})
    assert _lora_fwd(sh, lora(), sgu=FAKE, sdn=FAKE) == L.E_INVAL
    assert _lora_fwd(L.make_desc(**{**good, "dtype": L.F32}), lora()) == L.E_UNSUPPORTED
    need = lib.maskmoe_layer_lora_workspace_bytes(ctypes.byref(desc))
    assert need > lib.maskmoe_layer_workspace_bytes(ctypes.byref(desc))
    assert _lora_fwd(desc, lora(), ws_bytes=need - 1) == L.E_WORKSPACE
    # no tokens: nothing to do, whatever the adapters
    assert _lora_fwd(L.make_desc(**{**good, "T": 0}), lora(rank=99)) == L.OK


def test_lora_workspace_bytes_cover_the_adapter_buffers():
    lib = L.load()
    for (T, d, E, K, F, ns) in ((8192, 4096, 8, 2, 14336, 0), (4096, 2048, 64, 6, 1408, 2), (3, 256, 16, 4, 128, 1)):
        desc = L.make_desc(T, d, E, K, F, ns, L.BF16)
        base = lib.maskmoe_layer_workspace_bytes(ctypes.byref(desc))
        rows, G = T * (K + ns), E + ns
        extra = 2 * rows * 64 * 2 + G * (2 * F + d) * 64 * 2
        got = lib.maskmoe_layer_lora_workspace_bytes(ctypes.byref(desc))
        assert extra <= got - base <= extra + 4 * 256 and got % 256 == 0


def _offload(desc, B=4, policy=0, host=FAKE, ws_bytes=1 << 40, **kw):
    lib = L.load()
    a = dict(x=FAKE, w=FAKE, sgu=None, sdn=None, slots=FAKE, state=FAKE, y=FAKE, ws=FAKE)
    a.update(kw)
    return lib.maskmoe_offload_decode_step(ctypes.byref(desc), a["x"], a["w"], None, None, host, host, a["sgu"],
                                           a["sdn"], B, policy, a["slots"], a["slots"], a["state"], a["y"], None,
                                           None, None, None, a["ws"], ws_bytes, None, None)


def test_offload_step_rejects_invalid_arguments():
    lib = L.load()
    good = dict(T=1, d=128, E=8, K=2, F=256, n_shared=0, dtype=L.BF16, route_mode=L.ROUTE_PLAIN,
                gate_mode=L.GATE_RENORM)
    desc = L.make_desc(**good)
    assert _offload(L.make_desc(**{**good, "T": 2})) == L.E_UNSUPPORTED
    assert _offload(L.make_desc(**{**good, "dtype": L.F32})) == L.E_UNSUPPORTED
    assert _offload(L.make_desc(**{**good, "E": 65, "K": 2}), B=4) == L.E_UNSUPPORTED
    assert _offload(L.make_desc(**{**good, "d": 96})) == L.E_UNSUPPORTED
    assert _offload(desc, B=1) == L.E_INVAL           # B < K
    assert _offload(desc, B=9) == L.E_INVAL           # B > E
    assert _offload(desc, policy=3) == L.E_INVAL
    assert _offload(desc, state=None) == L.E_INVAL
    assert _offload(desc, slots=FAKE + 8) == L.E_INVAL
    assert _offload(desc, host=FAKE) == L.E_INVAL     # not pinned host memory
    assert _offload(L.make_desc(**{**good, "n_shared": 1})) == L.E_INVAL
    need = lib.maskmoe_offload_workspace_bytes(ctypes.byref(desc))
    assert need > lib.maskmoe_layer_workspace_bytes(ctypes.byref(desc))


def test_workspace_bytes_monotone_in_tokens():
    lib = L.load()
    for (d, E, K, F, ns, dt) in ((4096, 8, 2, 14336, 0, L.BF16), (2048, 64, 6, 1408, 2, L.BF16),
                                 (256, 8, 2, 512, 0, L.F32)):
        prev = 0
        for T in list(range(0, 40)) + [100, 1000, 8192]:
            desc = L.make_desc(T, d, E, K, F, ns, dt)
            b = lib.maskmoe_layer_workspace_bytes(ctypes.byref(desc))
            assert b >= prev and b % 256 == 0
            prev = b
    assert lib.maskmoe_layer_workspace_bytes(ctypes.byref(L.make_desc(-1, 64, 8, 2, 64))) == 0


def _cache(L_=1, S=1, N=4, K=2, E=8, B=4, policy=0, trace=FAKE, state=None, fetches=FAKE, hits=FAKE):
    lib = L.load()
    return lib.maskmoe_cache_fetches(trace, L_, S, N, K, E, B, policy, state, None, fetches, hits, None, None, None)


def test_cache_rejects_invalid_arguments():
    assert _cache(B=1) == L.E_INVAL          # B < K
    assert _cache(K=0) == L.E_INVAL
    assert _cache(K=9) == L.E_INVAL          # K > E
    assert _cache(N=-1) == L.E_INVAL
    assert _cache(policy=3) == L.E_INVAL
    assert _cache(policy=-1) == L.E_INVAL
    assert _cache(E=65, K=2) == L.E_UNSUPPORTED
    assert _cache(N=1 << 23, K=2) == L.E_UNSUPPORTED
    assert _cache(fetches=None) == L.E_INVAL
    assert _cache(trace=None) == L.E_INVAL
    assert _cache(L_=0, trace=None, fetches=None, hits=None) == L.OK   # nothing to do


def test_packed_layout_validation():
    """The packed weight layout: an unknown layout value is invalid; packed needs bf16,
    d % 128 == 0 and F % 64 == 0; the training and backward entry points refuse it."""
    lib = L.load()
    good = dict(T=32, d=128, E=8, K=2, F=256, n_shared=0, dtype=L.BF16, route_mode=L.ROUTE_PLAIN,
                gate_mode=L.GATE_RENORM, weight_layout=L.LAYOUT_PACKED)
    desc = L.make_desc(**good)
    assert lib.maskmoe_layer_workspace_bytes(ctypes.byref(desc)) > 0
    assert lib.maskmoe_layer_workspace_bytes(ctypes.byref(L.make_desc(**{**good, "weight_layout": 2}))) == 0
    assert _fwd(L.make_desc(**{**good, "weight_layout": 2}), ws_bytes=1 << 30) == L.E_INVAL
    assert _fwd(L.make_desc(**{**good, "weight_layout": -1}), ws_bytes=1 << 30) == L.E_INVAL
    assert _fwd(L.make_desc(**{**good, "dtype": L.F32}), ws_bytes=1 << 30) == L.E_UNSUPPORTED
    assert _fwd(L.make_desc(**{**good, "d": 192}), ws_bytes=1 << 30) == L.E_UNSUPPORTED
    assert _fwd(L.make_desc(**{**good, "F": 96}), ws_bytes=1 << 30) == L.E_UNSUPPORTED
    assert _fwd(L.make_desc(**{**good, "weight_layout": L.LAYOUT_ROWS, "d": 192}), ws_bytes=0) == L.E_WORKSPACE
    assert lib.maskmoe_layer_forward_train(ctypes.byref(desc), FAKE, FAKE, None, None, FAKE, FAKE, None, None, FAKE,
                                           FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 40, None) == L.E_UNSUPPORTED
    assert lib.maskmoe_layer_backward(ctypes.byref(desc), FAKE, FAKE, FAKE, None, None, FAKE, FAKE, FAKE, 1 << 40,
                                      FAKE, FAKE, FAKE, None, None, FAKE, 1 << 40, None) == L.E_UNSUPPORTED
    assert _offload(L.make_desc(**{**good, "T": 1, "d": 192})) == L.E_UNSUPPORTED
    assert _offload(L.make_desc(**{**good, "T": 1})) == L.E_INVAL     # accepted; FAKE is not pinned host memory


def test_pack_rejects_invalid_arguments():
    lib = L.load()
    pack = lambda desc, n=2, gu=FAKE, dn=FAKE, pgu=FAKE + 0x1000, pdn=FAKE + 0x2000: lib.maskmoe_pack_expert_weights(
        ctypes.byref(desc), n, gu, dn, pgu, pdn, None)
    desc = L.make_desc(T=0, d=256, E=1, K=1, F=128)
    assert pack(desc, n=0) == L.OK                                    # nothing to do, nothing launched
    assert pack(desc, n=-1) == L.E_INVAL
    assert pack(desc, pgu=None) == L.E_INVAL                          # source without destination
    assert pack(desc, gu=None) == L.E_INVAL                           # destination without source
    assert pack(desc, pdn=FAKE) == L.E_INVAL                          # in place
    assert pack(desc, gu=FAKE + 8) == L.E_INVAL                       # misaligned
    assert pack(L.make_desc(T=0, d=256, E=1, K=1, F=128, dtype=L.F32)) == L.E_UNSUPPORTED
    assert pack(L.make_desc(T=0, d=192, E=1, K=1, F=128)) == L.E_UNSUPPORTED
    assert pack(L.make_desc(T=0, d=256, E=1, K=1, F=96)) == L.E_UNSUPPORTED
    assert pack(L.make_desc(T=0, d=0, E=1, K=1, F=128)) == L.E_INVAL
