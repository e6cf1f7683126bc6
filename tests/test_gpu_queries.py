"""Several queries over one video in one wz_condense_queries call: each
query's outputs must be bitwise those of wz_condense with that query alone,
and (at the parity bar) the oracle's.  Covers the shared pass over X (bf16,
queries x Q <= 64: query columns split across 16-column MFMA tiles, a query
boundary inside a tile; groups of queries sharing several passes, the last
group smaller) and the separate passes otherwise.  Marked gpu."""
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


def _bits(t):
    return t.view(torch.int16) if t.dtype == torch.bfloat16 else t


def _queries(q, n):
    """n different queries of one shape derived from q: rotated channels,
    reversed tokens, negated."""
    out = [q, q.roll(8, dims=-1), q.flip(0), -q, q.roll(24, dims=-1), -q.flip(0), q.roll(40, dims=-1),
           -q.roll(8, dims=-1)]
    return torch.stack([x.contiguous() for x in out[:n]])


QCASES = {
    "q20_x3": dict(T=6, H=5, W=7, C=136, Q=20, B=50),  # 60 columns, query 1 starts inside a tile
    "q40_x2": dict(T=5, H=4, W=6, C=72, Q=40, B=30),   # 80 columns: separate passes
}


def _case(name):
    if name in EDGE:
        return _random_case(0, **EDGE[name])
    if name in QCASES:
        return _random_case(3000, **QCASES[name])
    return G.workload_case(name)


@pytest.mark.parametrize("name,n,out_dtype", [("t64_14x14_c3584", 2, wz.WZ_BF16), ("t32_14x14_c3584", 4, wz.WZ_F32),
                                              ("odd_3x5", 3, wz.WZ_F32), ("q20_x3", 3, wz.WZ_F32),
                                              ("small_query_bf16", 8, wz.WZ_BF16), ("q40_x2", 2, wz.WZ_F32),
                                              ("tiny", 3, wz.WZ_F32), ("t128_13x13_c3584", 2, wz.WZ_F32),
                                              ("t256_27x27_c1152", 2, wz.WZ_BF16),
                                              # several passes over X, each shared by a group of queries
                                              ("t64_14x14_c3584", 4, wz.WZ_BF16), ("odd_3x5", 5, wz.WZ_F32),
                                              ("q20_x3", 5, wz.WZ_F32)])
def test_condense_queries_matches_single(name, n, out_dtype):
    wl, inp, out = _case(name)
    p = wz.problem_of(wl, out_dtype)
    X, q0 = wz.to_device(inp, DEV)
    qs = _queries(q0, n)
    print(f"[case] queries {name} T={wl.T} {wl.H}x{wl.W} C={wl.C} Q={wl.Q} B={wl.B} G={n}", flush=True)
    ws = torch.empty(n * wz.workspace_bytes(p), dtype=torch.uint8, device=DEV)
    ws.fill_(0x5A)  # contents on entry are ignored
    tok, idx, b, o = wz.condense_queries(p, X, qs, ws=ws)
    singles = [wz.condense(p, X, qs[g]) for g in range(n)]
    torch.cuda.synchronize()
    for g, (t1, i1, b1, o1) in enumerate(singles):
        k = int(o1[-1])
        assert torch.equal(b[g], b1) and torch.equal(o[g], o1), g
        assert torch.equal(idx[g][:k], i1[:k]), g
        assert torch.equal(_bits(tok[g][:k]), _bits(t1[:k])), g
    # query 0 is the case's own query: the oracle's outputs
    k = int(out["offset"][-1])
    assert np.array_equal(b[0].cpu().numpy(), out["budget"])
    assert np.array_equal(idx[0][:k].cpu().numpy(), out["index"])
    tol = G.tol_for(wl.dtype) if out_dtype == wz.WZ_F32 else G.TOL_BF16_OUT
    assert G.within(tok[0][:k].float().cpu().numpy(), out["tokens"], tol)


def test_condense_queries_oracle_every_query():
    """Every query of a shared pass against the oracle run on that query."""
    wl, inp, _ = _case("q20_x3")
    p = wz.problem_of(wl)
    X, q0 = wz.to_device(inp, DEV)
    qs = _queries(q0, 3)
    tok, idx, b, o = wz.condense_queries(p, X, qs)
    torch.cuda.synchronize()
    Xf = inp.X_f64()
    for g in range(3):
        qg = qs[g].float().cpu().numpy().astype(np.float64)
        ref = oracle.condense(Xf, qg, wl.B, wl.levels, wl.lam, wl.tau)
        if G.check_margins(ref, wl.N, wl.B, wl.tau):
            continue  # a decision within the margin: the bitwise comparison above covers this query
        k = int(ref["offset"][-1])
        assert np.array_equal(b[g].cpu().numpy(), ref["budget"]), g
        assert np.array_equal(idx[g][:k].cpu().numpy(), ref["index"]), g
        assert G.within(tok[g][:k].cpu().numpy(), ref["tokens"], G.tol_for(wl.dtype)), g


@pytest.mark.parametrize("name,sb,n", [("t64_14x14_c3584", wz.WZ_DB4, 2), ("split_32x32_c200", wz.WZ_BIOR44, 3)])
def test_condense_queries_filter_bank_matches_single(name, sb, n):
    """With a db4 / bior4.4 spatial basis (the fused kernel at 14x14, the split form with its rows in the
    workspace on a large bf16 grid) each query's outputs are bitwise those of its single call."""
    if name == "split_32x32_c200":
        wl, inp, _ = _random_case(0, T=3, H=32, W=32, C=200, Q=16, B=300)
    else:
        wl, inp, _ = _case(name)
    p = wz.problem_of(wl, wz.WZ_BF16, spatial_basis=sb)
    X, q0 = wz.to_device(inp, DEV)
    qs = _queries(q0, n)
    tok, idx, b, o = wz.condense_queries(p, X, qs)
    singles = [wz.condense(p, X, qs[g]) for g in range(n)]
    torch.cuda.synchronize()
    for g, (t1, i1, b1, o1) in enumerate(singles):
        k = int(o1[-1])
        assert k > 0
        assert torch.equal(b[g], b1) and torch.equal(o[g], o1), g
        assert torch.equal(idx[g][:k], i1[:k]), g
        assert torch.equal(_bits(tok[g][:k]), _bits(t1[:k])), g
