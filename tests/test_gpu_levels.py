"""The two-level spatial Haar modulator (cfg.spatial_levels = 2, selection) on
the GPU against the oracle: budgets and indices bit-exact, tokens at the parity
bar.  Marked gpu."""
import numpy as np
import pytest
import torch

import gpu_util as G
import libutil
import oracle
from test_gpu_parity import EDGE, _random_case
from paper_2607_23265_amd import wavezip as wz

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(scope="module", autouse=True)
def _lib():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    libutil.ensure_built()


def _case(name):
    wl, inp, _ = _random_case(0, **EDGE[name]) if name in EDGE else G.workload_case(name)
    out = oracle.condense(inp.X_f64(), inp.query_f64(), wl.B, wl.levels, wl.lam, float(np.float32(wl.tau)),
                          spatial_levels=2)
    return wl, inp, out


def _np(t):
    return t.detach().float().cpu().numpy() if t.dtype in (torch.bfloat16, torch.float32) else t.cpu().numpy()


@pytest.mark.parametrize("name,out_dtype", [("tiny", wz.WZ_F32), ("t64_14x14_c3584", wz.WZ_BF16),
                                            ("t32_14x14_c3584", wz.WZ_BF16), ("t256_27x27_c1152", wz.WZ_BF16),
                                            ("t128_13x13_c3584", wz.WZ_F32), ("odd_3x5", wz.WZ_F32),
                                            ("single_token", wz.WZ_F32), ("row_1x7", wz.WZ_F32),
                                            ("col_7x1", wz.WZ_F32), ("many_frames", wz.WZ_F32)])
def test_condense_two_levels(name, out_dtype):
    wl, inp, out = _case(name)
    p = wz.problem_of(wl, out_dtype, spatial_levels=2)
    X, q = wz.to_device(inp, DEV)
    print(f"[case] two levels {name} T={wl.T} {wl.H}x{wl.W} C={wl.C} Q={wl.Q} B={wl.B}", flush=True)
    tok, idx, b, o = wz.condense(p, X, q)
    torch.cuda.synchronize()
    n = int(out["offset"][-1])
    assert np.array_equal(_np(b), out["budget"]) and np.array_equal(_np(o), out["offset"])
    assert np.array_equal(_np(idx)[:n], out["index"])
    tol = G.tol_for(wl.dtype) if out_dtype == wz.WZ_F32 else G.TOL_BF16_OUT
    assert G.within(_np(tok)[:n], out["tokens"], tol, f"{wl.name} two-level tokens")


@pytest.mark.parametrize("name", ["tiny", "t64_14x14_c3584", "odd_3x5"])
def test_stage_spatial_two_levels(name):
    """wz_spatial_dwt_condense with two levels, fed the oracle's scores and offsets (gates formed in-kernel)."""
    wl, inp, out = _case(name)
    p = wz.problem_of(wl, wz.WZ_F32, spatial_levels=2)
    X, _ = wz.to_device(inp, DEV)
    a = torch.from_numpy(out["a"].astype(np.float32).ravel()).to(DEV)
    off = torch.from_numpy(out["offset"].astype(np.int32)).to(DEV)
    tok, idx = wz.spatial_dwt_condense(p, X, a, off)
    torch.cuda.synchronize()
    n = int(out["offset"][-1])
    assert np.array_equal(_np(idx)[:n], out["index"])
    assert G.within(_np(tok)[:n], out["tokens"], G.tol_for(wl.dtype))
