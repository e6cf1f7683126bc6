"""wz_condense_noalloc (static device scratch, no workspace) against wz_condense.

Called through the C ABI on the GPU.  Two calls in a row on the same device
share the static array: the first on the benchmark-sized workload, the second
on a smaller one, so the second starts from whatever the first left there.
Each call's budgets, offsets and kept-token indices must equal wz_condense's
on the same inputs bit for bit, and its tokens too (the same kernels run on
the same inputs); the oracle checks the small case as well.
"""
import ctypes

import numpy as np
import pytest
import torch

import gpu_util as G
import libutil
from paper_2607_23265_amd import synth
from paper_2607_23265_amd import wavezip as wz

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


@pytest.fixture(scope="module", autouse=True)
def _lib():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    libutil.ensure_built()


def _np(t):
    return t.detach().float().cpu().numpy() if t.dtype in (torch.bfloat16, torch.float32) else t.cpu().numpy()


def _both(p, X, q):
    ref = wz.condense(p, X, q)
    got = wz.condense_noalloc(p, X, q)
    torch.cuda.synchronize()
    return ref, got


def _same(ref, got):
    for a, b in zip(ref, got):
        assert torch.equal(a, b)


def test_two_calls_second_smaller():
    big = synth.WORKLOADS["t64_14x14_c3584"]
    small = synth.small("t64_14x14_c3584", T=8, C=256, Q=16, B=157)
    for wl, out_dtype in ((big, wz.WZ_BF16), (small, wz.WZ_F32)):
        print(f"[case] noalloc {wl.name} T={wl.T} C={wl.C} Q={wl.Q} B={wl.B}", flush=True)
        inp = synth.generate(wl)
        p = wz.problem_of(wl, out_dtype)
        assert wz.workspace_bytes(p) <= wz.lib().wz_noalloc_scratch_bytes()
        X, q = wz.to_device(inp, DEV)
        ref, got = _both(p, X, q)
        _same(ref, got)
    # the small case against the oracle as well
    import oracle
    want = oracle.condense(inp.X_f64(), inp.query_f64(), small.B, small.levels, small.lam, small.tau)
    tok, idx, b, o = got
    n = int(want["offset"][-1])
    if not G.check_margins(want, small.N, small.B, small.tau):
        assert np.array_equal(_np(b), want["budget"]) and np.array_equal(_np(idx)[:n], want["index"])
        assert G.within(_np(tok)[:n], want["tokens"], G.TOL_F32_IN if small.dtype == "f32" else G.TOL_BF16_IN)


def test_filter_rows_beyond_scratch_use_the_fused_form():
    """db4 on a large bf16 grid with most tokens kept: the operator rows alone would not fit the scratch,
    so the call forms them in LDS (the fused form); its outputs equal wz_condense's (which has them in its
    workspace) bit for bit."""
    wl = synth.Workload("noalloc_split_T20_27x27", T=20, H=27, W=27, C=256, Q=16, dtype="bf16", B=14000)
    p = wz.problem_of(wl, wz.WZ_BF16, spatial_basis=wz.WZ_DB4)
    assert wz.workspace_bytes(p) > wz.lib().wz_noalloc_scratch_bytes()
    print(f"[case] noalloc {wl.name} T={wl.T} C={wl.C} Q={wl.Q} B={wl.B} db4", flush=True)
    X, q = wz.to_device(synth.generate(wl), DEV)
    ref, got = _both(p, X, q)
    assert int(ref[3][-1]) > 0
    _same(ref, got)


def test_rejects_problem_beyond_scratch():
    L = wz.lib()
    p = wz.Problem(T=2048, H=14, W=14, C=3584, Q=32, B=1000)
    assert wz.workspace_bytes(p) > L.wz_noalloc_scratch_bytes()
    cfg = p.config()
    fake = ctypes.c_void_p(0x10000)
    assert L.wz_condense_noalloc(ctypes.byref(cfg), fake, fake, fake, fake, None, None, None) == 9
    assert L.wz_status_str(9).decode().startswith("WZ_ERR_SCRATCH")
