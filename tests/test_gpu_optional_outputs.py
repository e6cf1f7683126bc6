"""wz_condense and wz_condense_batch with the optional budget and offset outputs
left NULL (the library then keeps them in the workspace): the kept tokens and
their indices are bitwise those of the same call with the outputs given, and
the given outputs are valid budgets, on every path that computes the budgets
(inside the selection kernel up to 256 frames, the budget kernel above; inside
the filter-bank modulator up to 64 frames, the budget kernel above, fused and
split forms).  Marked gpu."""
import ctypes

import numpy as np
import pytest
import torch

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


CASES = [
    # name, shape, spatial basis
    ("haar_T8", dict(T=8, H=6, W=6, C=64, Q=16, B=60), wz.WZ_HAAR),
    ("haar_T100_filter", dict(T=100, H=4, W=4, C=64, Q=16, B=600, tau=1.0), wz.WZ_HAAR),
    ("haar_T300", dict(T=300, H=3, W=3, C=32, Q=16, B=900), wz.WZ_HAAR),
    ("db4_T8", dict(T=8, H=6, W=6, C=64, Q=16, B=60), wz.WZ_DB4),
    ("bior_T100", dict(T=100, H=4, W=4, C=64, Q=16, B=600), wz.WZ_BIOR44),
    ("db4_split_T3", dict(T=3, H=32, W=32, C=200, Q=16, B=300), wz.WZ_DB4),
]


def _inputs(seed, T, H, W, C, Q, B, tau=0.0):
    wl = synth.Workload(f"opt_T{T}_{H}x{W}_C{C}", T=T, H=H, W=W, C=C, Q=Q, dtype="bf16", B=B, levels=2, lam=1.5,
                        tau=tau)
    rng = np.random.default_rng(seed)
    X = synth.f32_to_bf16_bits(rng.standard_normal((T, H, W, C)).astype(np.float32))
    q = synth.f32_to_bf16_bits((rng.standard_normal((Q, C)) / np.sqrt(C)).astype(np.float32))
    return wl, synth.Inputs(wl=wl, X=X, query=q)


def _call(fn, p, V, X, q, outputs):
    """One wz_condense (V = 0) or wz_condense_batch (V videos) call; budget and offset given or NULL."""
    n = max(V, 1)
    ws = torch.zeros(n * wz.workspace_bytes(p), dtype=torch.uint8, device=DEV)
    tok = torch.zeros((n, max(p.B, 1), p.C), dtype=torch.bfloat16, device=DEV)
    idx = torch.full((n, max(p.B, 1)), -1, dtype=torch.int32, device=DEV)
    b = torch.full((n, p.T), -1, dtype=torch.int32, device=DEV) if outputs else None
    o = torch.full((n, p.T + 1), -1, dtype=torch.int32, device=DEV) if outputs else None
    cfg = p.config()
    args = [wz._ptr(X), wz._ptr(q), wz._ptr(tok), wz._ptr(idx), wz._ptr(b), wz._ptr(o), wz._ptr(ws), ws.numel(),
            wz._stream(X.device)]
    st = fn(ctypes.byref(cfg), *args) if V == 0 else fn(ctypes.byref(cfg), V, *args)
    assert st == 0, wz.lib().wz_status_str(st)
    torch.cuda.synchronize()
    return tok, idx, b, o


@pytest.mark.parametrize("name,shape,sb", CASES)
def test_null_budget_and_offset(name, shape, sb):
    wl, inp = _inputs(7, **shape)
    print(f"[case] optional outputs {name} T={wl.T} {wl.H}x{wl.W} C={wl.C} B={wl.B} spatial={sb}", flush=True)
    p = wz.problem_of(wl, wz.WZ_BF16, spatial_basis=sb)
    X, q = wz.to_device(inp, DEV)
    L = wz.lib()
    tok1, idx1, b1, o1 = _call(L.wz_condense, p, 0, X, q, True)
    tok0, idx0, _, _ = _call(L.wz_condense, p, 0, X, q, False)
    b, o = b1[0].cpu().numpy(), o1[0].cpu().numpy()
    # valid budgets: non-negative, at most a frame's tokens, offsets their running sum, B in all
    assert (b >= 0).all() and (b <= wl.N).all()
    assert o[0] == 0 and np.array_equal(np.diff(o), b)
    # B in all, unless the frame filter leaves fewer tokens
    assert o[-1] == min(wl.B, wl.T * wl.N) if wl.tau == 0 else 0 < o[-1] <= wl.B
    n = int(o[-1])
    assert torch.equal(idx0[0, :n], idx1[0, :n])
    assert torch.equal(tok0[0, :n].view(torch.int16), tok1[0, :n].view(torch.int16))

    # two videos in one batch call, outputs NULL, against the single calls
    X2 = X.flip(0).contiguous()
    tokb, idxb, _, _ = _call(L.wz_condense_batch, p, 2, torch.stack([X, X2]), torch.stack([q, q]), False)
    tok2, idx2, _, o2 = _call(L.wz_condense, p, 0, X2, q, True)
    n2 = int(o2[0, -1])
    assert torch.equal(idxb[0, :n], idx1[0, :n]) and torch.equal(idxb[1, :n2], idx2[0, :n2])
    assert torch.equal(tokb[0, :n].view(torch.int16), tok1[0, :n].view(torch.int16))
    assert torch.equal(tokb[1, :n2].view(torch.int16), tok2[0, :n2].view(torch.int16))
