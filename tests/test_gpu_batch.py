"""Several videos in one wz_condense_batch call: each video's outputs must be
bitwise those of wz_condense on that video alone (and, for the first video,
the oracle's at the parity bar).  Marked gpu."""
import numpy as np
import pytest
import torch

import gpu_util as G
import libutil
from test_gpu_parity import EDGE, _random_case
from paper_2607_23265_amd import wavezip as wz

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(scope="module", autouse=True)
def _lib():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    libutil.ensure_built()


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t


def _videos(X, q):
    """Three different videos of one shape: the input, its frames reversed, and
    its channels rotated (query rotated alike)."""
    return ([X, X.flip(0).contiguous(), X.roll(8, dims=-1).contiguous()],
            [q, q.flip(0).contiguous(), q.roll(8, dims=-1).contiguous()])


def _case(name):
    if name in EDGE:
        return _random_case(0, **EDGE[name])
    return G.workload_case(name)


@pytest.mark.parametrize("name,out_dtype", [("tiny", wz.WZ_F32), ("t64_14x14_c3584", wz.WZ_BF16),
                                            ("t32_14x14_c3584", wz.WZ_BF16), ("t256_27x27_c1152", wz.WZ_BF16),
                                            ("t128_13x13_c3584", wz.WZ_F32), ("odd_3x5", wz.WZ_F32),
                                            ("many_frames", wz.WZ_F32)])
def test_condense_batch_matches_single(name, out_dtype):
    wl, inp, out = _case(name)
    p = wz.problem_of(wl, out_dtype)
    X0, q0 = wz.to_device(inp, DEV)
    Xs, qs = _videos(X0, q0)
    print(f"[case] batch {name} T={wl.T} {wl.H}x{wl.W} C={wl.C} Q={wl.Q} B={wl.B} V={len(Xs)}", flush=True)
    ws = torch.empty(len(Xs) * wz.workspace_bytes(p), dtype=torch.uint8, device=DEV)
    ws.fill_(0x5A)  # contents on entry are ignored
    tok, idx, b, o = wz.condense_batch(p, torch.stack(Xs), torch.stack(qs), ws=ws)
    singles = [wz.condense(p, x, q) for x, q in zip(Xs, qs)]
    torch.cuda.synchronize()
    for v, (t1, i1, b1, o1) in enumerate(singles):
        n = int(o1[-1])
        assert torch.equal(b[v], b1) and torch.equal(o[v], o1), v
        assert torch.equal(idx[v][:n], i1[:n]), v
        assert torch.equal(_bits(tok[v][:n]), _bits(t1[:n])), v
    n = int(out["offset"][-1])
    assert np.array_equal(b[0].cpu().numpy(), out["budget"])
    assert np.array_equal(idx[0][:n].cpu().numpy(), out["index"])
    tol = G.tol_for(wl.dtype) if out_dtype == wz.WZ_F32 else G.TOL_BF16_OUT
    assert G.within(tok[0][:n].float().cpu().numpy(), out["tokens"], tol)


def test_condense_batch_single_video_equals_condense():
    wl, inp, _ = G.workload_case("t64_14x14_c3584")
    p = wz.problem_of(wl, wz.WZ_BF16)
    X, q = wz.to_device(inp, DEV)
    tok, idx, b, o = wz.condense_batch(p, X[None], q[None])
    t1, i1, b1, o1 = wz.condense(p, X, q)
    torch.cuda.synchronize()
    assert torch.equal(_bits(tok[0]), _bits(t1)) and torch.equal(idx[0], i1)
    assert torch.equal(b[0], b1) and torch.equal(o[0], o1)
