"""The C ABI: exported symbols, status strings and host-side validation (no GPU needed).

Every call here fails validation, which returns before any HIP call is made.
"""
import ctypes
import subprocess

import pytest

import libutil
from paper_2607_23265_amd import wavezip as wz

OK, NULL, ALIGN, SHAPE, DTYPE, PARAM, BUDGET, WORKSPACE = range(8)


@pytest.fixture(scope="module")
def L():
    return libutil.ensure_built()


def cfg(**kw):
    p = dict(T=64, H=14, W=14, C=3584, Q=32, B=1254, in_dtype=wz.WZ_BF16, out_dtype=wz.WZ_F32, levels=2,
             lam=1.5, tau=0.0)
    p.update(kw)
    return wz.Problem(**p).config()


def test_every_declared_symbol_is_exported(L):
    names = libutil.declared_functions()
    assert set(names) == set(wz.EXPORTS)
    dyn = subprocess.run(["nm", "-D", "--defined-only", wz.LIB_PATH], capture_output=True, text=True).stdout
    exported = {line.split()[-1] for line in dyn.splitlines() if line.strip()}
    for n in names:
        assert n in exported, n
        assert hasattr(L, n)


def test_status_strings(L):
    for code, name in wz._STATUS.items():
        assert L.wz_status_str(code).decode().startswith(name)
    assert L.wz_status_str(99) == b"unknown wz_status"


def test_config_struct_layout():
    assert ctypes.sizeof(wz.Config) == 64
    assert wz.Config.B.offset == 32 and wz.Config.lambda_.offset == 40 and wz.Config.tau.offset == 44
    assert wz.Config.assign.offset == 48 and wz.Config.spatial_levels.offset == 52
    assert wz.Config.temporal_basis.offset == 56 and wz.Config.spatial_basis.offset == 60


def test_workspace_bytes(L):
    small = L.wz_workspace_bytes(ctypes.byref(cfg(T=8)))
    big = L.wz_workspace_bytes(ctypes.byref(cfg()))
    assert 0 < small < big and big % 256 == 0
    assert L.wz_workspace_bytes(ctypes.byref(cfg(C=12))) == 0
    assert L.wz_workspace_bytes(None) == 0


@pytest.mark.parametrize("kw,code", [
    (dict(T=0), SHAPE), (dict(T=2049), SHAPE), (dict(H=0), SHAPE), (dict(H=65, W=64), SHAPE),
    (dict(Q=0), SHAPE), (dict(Q=1025), SHAPE), (dict(C=12), SHAPE), (dict(C=0), SHAPE),
    (dict(in_dtype=7), DTYPE), (dict(out_dtype=-1), DTYPE), (dict(levels=0), PARAM), (dict(levels=17), PARAM),
    (dict(lam=-1.0), PARAM), (dict(lam=float("inf")), PARAM), (dict(tau=2.5), PARAM), (dict(tau=float("nan")), PARAM),
    (dict(B=-1), BUDGET), (dict(B=64 * 196 + 1), BUDGET), (dict(assign=2), PARAM), (dict(assign=-1), PARAM),
    (dict(spatial_levels=3), PARAM), (dict(spatial_levels=-1), PARAM),
    (dict(spatial_levels=2, assign=1), PARAM),
    (dict(temporal_basis=3), PARAM), (dict(temporal_basis=-1), PARAM), (dict(spatial_basis=3), PARAM),
    (dict(spatial_basis=1, assign=1), PARAM), (dict(spatial_basis=2, spatial_levels=2), PARAM),
    (dict(spatial_basis=1, H=65, W=2), SHAPE), (dict(spatial_basis=2, H=40, W=40, B=10), SHAPE),
])
def test_invalid_config(L, kw, code):
    c = cfg(**kw)
    fake = ctypes.c_void_p(0x10000)
    assert L.wz_relevance(ctypes.byref(c), fake, fake, fake, fake, fake, fake, 1 << 30, None) == code
    assert L.wz_relevance_pass(ctypes.byref(c), fake, fake, fake, fake, 1 << 30, None) == code
    assert L.wz_temporal_budget(ctypes.byref(c), fake, fake, fake, fake, None, None) == code
    assert L.wz_spatial_dwt_condense(ctypes.byref(c), fake, fake, fake, fake, fake, None) == code
    assert L.wz_condense(ctypes.byref(c), fake, fake, fake, fake, None, None, fake, 1 << 30, None) == code
    assert L.wz_condense_batch(ctypes.byref(c), 2, fake, fake, fake, fake, None, None, fake, 1 << 30, None) == code
    assert L.wz_condense_queries(ctypes.byref(c), 2, fake, fake, fake, fake, None, None, fake, 1 << 30, None) == code


def test_pointer_checks(L):
    c = cfg()
    ok = ctypes.c_void_p(0x10000)
    odd = ctypes.c_void_p(0x10008)     # 8-byte aligned, not 16
    odd4 = ctypes.c_void_p(0x10002)
    nul = ctypes.c_void_p(0)
    need = L.wz_workspace_bytes(ctypes.byref(c))
    assert L.wz_relevance(None, ok, ok, ok, ok, ok, ok, need, None) == NULL
    assert L.wz_relevance(ctypes.byref(c), nul, ok, ok, ok, ok, ok, need, None) == NULL
    assert L.wz_relevance(ctypes.byref(c), odd, ok, ok, ok, ok, ok, need, None) == ALIGN
    assert L.wz_relevance(ctypes.byref(c), ok, odd, ok, ok, ok, ok, need, None) == ALIGN
    assert L.wz_relevance(ctypes.byref(c), ok, ok, odd4, ok, ok, ok, need, None) == ALIGN
    assert L.wz_relevance(ctypes.byref(c), ok, ok, ok, ok, ok, nul, need, None) == NULL
    assert L.wz_relevance(ctypes.byref(c), ok, ok, ok, ok, ok, ok, need - 1, None) == WORKSPACE
    assert L.wz_relevance(ctypes.byref(c), ok, ok, ok, ok, ok, ctypes.c_void_p(0x10010), need, None) == WORKSPACE
    assert L.wz_relevance_pass(None, ok, ok, ok, ok, need, None) == NULL
    assert L.wz_relevance_pass(ctypes.byref(c), nul, ok, ok, ok, need, None) == NULL
    assert L.wz_relevance_pass(ctypes.byref(c), ok, odd, ok, ok, need, None) == ALIGN
    assert L.wz_relevance_pass(ctypes.byref(c), ok, ok, odd4, ok, need, None) == ALIGN
    assert L.wz_relevance_pass(ctypes.byref(c), ok, ok, ok, nul, need, None) == NULL
    assert L.wz_relevance_pass(ctypes.byref(c), ok, ok, ok, ok, need - 1, None) == WORKSPACE
    assert L.wz_relevance_pass(ctypes.byref(c), ok, ok, ok, ctypes.c_void_p(0x10010), need, None) == WORKSPACE
    assert L.wz_temporal_budget(ctypes.byref(c), ok, ok, nul, ok, None, None) == NULL
    assert L.wz_temporal_budget(ctypes.byref(c), ok, ok, ok, odd4, None, None) == ALIGN
    assert L.wz_temporal_budget(ctypes.byref(c), ok, ok, ok, ok, odd4, None) == ALIGN
    assert L.wz_spatial_dwt_condense(ctypes.byref(c), ok, ok, ok, odd, ok, None) == ALIGN
    assert L.wz_spatial_dwt_condense(ctypes.byref(c), ok, ok, ok, ok, nul, None) == NULL
    assert L.wz_spatial_dwt_condense(ctypes.byref(c), ok, ok, nul, ok, ok, None) == NULL
    assert L.wz_spatial_dwt_condense(ctypes.byref(c), nul, ok, ok, ok, ok, None) == NULL
    assert L.wz_condense(ctypes.byref(c), ok, ok, nul, ok, None, None, ok, need, None) == NULL
    assert L.wz_condense(ctypes.byref(c), ok, ok, ok, ok, odd4, None, ok, need, None) == ALIGN
    assert L.wz_condense(ctypes.byref(c), ok, ok, ok, ok, None, None, ok, need - 256, None) == WORKSPACE
    assert L.wz_condense_batch(ctypes.byref(c), 0, ok, ok, ok, ok, None, None, ok, need, None) == SHAPE
    assert L.wz_condense_batch(ctypes.byref(c), 9, ok, ok, ok, ok, None, None, ok, 9 * need, None) == SHAPE
    assert L.wz_condense_batch(ctypes.byref(c), 3, ok, ok, ok, ok, None, None, ok, 3 * need - 1, None) == WORKSPACE
    assert L.wz_condense_batch(ctypes.byref(c), 3, nul, ok, ok, ok, None, None, ok, 3 * need, None) == NULL
    assert L.wz_condense_batch(ctypes.byref(c), 3, ok, ok, ok, odd4, None, None, ok, 3 * need, None) == ALIGN
    assert L.wz_condense_queries(ctypes.byref(c), 0, ok, ok, ok, ok, None, None, ok, need, None) == SHAPE
    assert L.wz_condense_queries(ctypes.byref(c), 9, ok, ok, ok, ok, None, None, ok, 9 * need, None) == SHAPE
    assert L.wz_condense_queries(ctypes.byref(c), 3, ok, ok, ok, ok, None, None, ok, 3 * need - 1, None) == WORKSPACE
    assert L.wz_condense_queries(ctypes.byref(c), 3, ok, nul, ok, ok, None, None, ok, 3 * need, None) == NULL
    assert L.wz_condense_queries(ctypes.byref(c), 3, ok, ok, ok, odd4, None, None, ok, 3 * need, None) == ALIGN


def test_binding_refuses_cpu_tensors():
    import torch
    p = wz.Problem(T=2, H=2, W=2, C=8, Q=1, B=2)
    with pytest.raises(ValueError):
        wz.relevance(p, torch.zeros(2, 2, 2, 8), torch.zeros(1, 8))
