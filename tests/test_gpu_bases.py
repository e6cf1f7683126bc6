"""db4 and bior4.4 wavelet bases (cfg.temporal_basis / cfg.spatial_basis) on the
GPU against the oracle's filter banks: budgets, offsets and kept-token indices
bit-exact, tokens at the parity bar.  Marked gpu.

The workloads' seeds were chosen for the Haar transforms; with a longer
temporal basis their budgets change, and on the 27x27 workload a few frames'
selection boundaries then fall inside the tie margin.  There the budgets and
offsets still compare exactly, and indices and tokens on every frame that
clears the margin (the frames that do not are listed by the margin check).
"""
import numpy as np
import pytest
import torch

import gpu_util as G
import libutil
import margins
import oracle
from test_gpu_parity import EDGE, _random_case
from paper_2607_23265_amd import synth
from paper_2607_23265_amd import wavezip as wz

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
NAMES = {wz.WZ_HAAR: "haar", wz.WZ_DB4: "db4", wz.WZ_BIOR44: "bior4.4"}


@pytest.fixture(scope="module", autouse=True)
def _lib():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    libutil.ensure_built()


def _np(t):
    return t.detach().float().cpu().numpy() if t.dtype in (torch.bfloat16, torch.float32) else t.cpu().numpy()


# the edge cases of the parity tests, plus the largest grids the filter banks
# take; with bf16 inputs on large grids the operator rows are formed once per
# frame and contracted by a second kernel (the split form): a ragged channel
# count (a partly filled wave), several 48-row sweeps per frame, and two
# balanced channel slices of 640 and 512 channels
CASE_EDGE = dict(EDGE, grid_32x32=dict(T=3, H=32, W=32, C=96, Q=16, B=300),
                 grid_16x64=dict(T=2, H=16, W=64, C=72, Q=16, B=200),
                 split_32x32_c200=dict(T=3, H=32, W=32, C=200, Q=16, B=300),
                 split_27x27_c1152=dict(T=2, H=27, W=27, C=1152, Q=16, B=420))


def _case(name, tb, sb):
    wl, inp, _ = _random_case(0, **CASE_EDGE[name]) if name in CASE_EDGE else G.workload_case(name)
    out = oracle.condense(inp.X_f64(), inp.query_f64(), wl.B, wl.levels, wl.lam, float(np.float32(wl.tau)),
                          temporal_basis=NAMES[tb], spatial_basis=NAMES[sb])
    return wl, inp, out


def _undecidable_frames(out, wl):
    """Frames whose selection boundary is within the tie margin (nothing else may be)."""
    bad = G.check_margins(out, wl.N, wl.B, wl.tau)
    assert all(kind == "selection" for kind, _ in bad), bad
    return {detail[0] for _, detail in bad}


def _compare(wl, out, tok, idx, b, o, tol, skip=frozenset()):
    n = int(out["offset"][-1])
    assert np.array_equal(_np(b), out["budget"]) and np.array_equal(_np(o), out["offset"])
    rows = np.ones(n, dtype=bool)
    for t in skip:
        rows[out["offset"][t]:out["offset"][t + 1]] = False
    assert np.array_equal(_np(idx)[:n][rows], out["index"][rows])
    assert G.within(_np(tok)[:n][rows], out["tokens"][rows], tol)


CASES = [
    # workload, temporal basis, spatial basis, output dtype
    ("tiny", wz.WZ_DB4, wz.WZ_DB4, wz.WZ_F32),
    ("tiny", wz.WZ_BIOR44, wz.WZ_BIOR44, wz.WZ_F32),
    ("tiny", wz.WZ_HAAR, wz.WZ_BIOR44, wz.WZ_F32),
    ("t32_14x14_c3584", wz.WZ_BIOR44, wz.WZ_DB4, wz.WZ_BF16),
    ("t64_14x14_c3584", wz.WZ_HAAR, wz.WZ_DB4, wz.WZ_BF16),
    ("t64_14x14_c3584", wz.WZ_HAAR, wz.WZ_BIOR44, wz.WZ_F32),
    ("t64_14x14_c3584", wz.WZ_DB4, wz.WZ_HAAR, wz.WZ_BF16),
    ("t64_14x14_c3584", wz.WZ_BIOR44, wz.WZ_HAAR, wz.WZ_BF16),
    ("t128_13x13_c3584", wz.WZ_BIOR44, wz.WZ_DB4, wz.WZ_BF16),
    ("t256_27x27_c1152", wz.WZ_HAAR, wz.WZ_BIOR44, wz.WZ_BF16),
    ("t256_27x27_c1152", wz.WZ_DB4, wz.WZ_HAAR, wz.WZ_BF16),
    ("odd_3x5", wz.WZ_DB4, wz.WZ_DB4, wz.WZ_F32),
    ("row_1x7", wz.WZ_BIOR44, wz.WZ_BIOR44, wz.WZ_F32),
    ("col_7x1", wz.WZ_DB4, wz.WZ_BIOR44, wz.WZ_F32),
    ("single_token", wz.WZ_BIOR44, wz.WZ_DB4, wz.WZ_F32),
    ("single_frame", wz.WZ_DB4, wz.WZ_DB4, wz.WZ_F32),
    ("budget_zero", wz.WZ_DB4, wz.WZ_DB4, wz.WZ_F32),
    ("budget_one", wz.WZ_BIOR44, wz.WZ_BIOR44, wz.WZ_F32),
    ("budget_all", wz.WZ_DB4, wz.WZ_BIOR44, wz.WZ_F32),
    ("ragged_channels", wz.WZ_DB4, wz.WZ_DB4, wz.WZ_F32),
    ("min_channels", wz.WZ_BIOR44, wz.WZ_DB4, wz.WZ_F32),
    ("fp32_query32", wz.WZ_DB4, wz.WZ_BIOR44, wz.WZ_F32),
    ("levels_4", wz.WZ_BIOR44, wz.WZ_DB4, wz.WZ_F32),
    ("odd_T_levels_2", wz.WZ_DB4, wz.WZ_BIOR44, wz.WZ_F32),
    ("frame_filter", wz.WZ_BIOR44, wz.WZ_DB4, wz.WZ_F32),
    ("lambda_zero", wz.WZ_DB4, wz.WZ_DB4, wz.WZ_F32),
    ("many_frames", wz.WZ_HAAR, wz.WZ_BIOR44, wz.WZ_F32),
    ("max_channels", wz.WZ_HAAR, wz.WZ_DB4, wz.WZ_F32),
    ("query_128_passes", wz.WZ_BIOR44, wz.WZ_BIOR44, wz.WZ_BF16),
    ("grid_32x32", wz.WZ_DB4, wz.WZ_DB4, wz.WZ_F32),
    ("grid_16x64", wz.WZ_BIOR44, wz.WZ_BIOR44, wz.WZ_F32),
    ("t256_27x27_c1152", wz.WZ_HAAR, wz.WZ_DB4, wz.WZ_F32),
    ("split_32x32_c200", wz.WZ_HAAR, wz.WZ_DB4, wz.WZ_BF16),
    ("split_32x32_c200", wz.WZ_BIOR44, wz.WZ_BIOR44, wz.WZ_F32),
    ("split_27x27_c1152", wz.WZ_HAAR, wz.WZ_BIOR44, wz.WZ_BF16),
    # Haar temporal basis with a filter-bank spatial basis at T <= 64: the budgets
    # inside the modulator's first kernel (fused form, the split form's row
    # kernel): frames that keep nothing, every token, one frame, the frame
    # filter, several levels, fp32 inputs, lambda = 0, one-token frames
    ("budget_zero", wz.WZ_HAAR, wz.WZ_DB4, wz.WZ_F32),
    ("budget_one", wz.WZ_HAAR, wz.WZ_BIOR44, wz.WZ_F32),
    ("budget_all", wz.WZ_HAAR, wz.WZ_DB4, wz.WZ_F32),
    ("single_frame", wz.WZ_HAAR, wz.WZ_BIOR44, wz.WZ_F32),
    ("frame_filter", wz.WZ_HAAR, wz.WZ_DB4, wz.WZ_F32),
    ("levels_4", wz.WZ_HAAR, wz.WZ_BIOR44, wz.WZ_F32),
    ("odd_T_levels_2", wz.WZ_HAAR, wz.WZ_DB4, wz.WZ_F32),
    ("fp32_query32", wz.WZ_HAAR, wz.WZ_DB4, wz.WZ_F32),
    ("lambda_zero", wz.WZ_HAAR, wz.WZ_BIOR44, wz.WZ_F32),
    ("single_token", wz.WZ_HAAR, wz.WZ_DB4, wz.WZ_F32),
    ("t32_14x14_c3584", wz.WZ_HAAR, wz.WZ_BIOR44, wz.WZ_BF16),
    ("split_32x32_c200", wz.WZ_HAAR, wz.WZ_BIOR44, wz.WZ_F32),
    # above 64 frames (the budget kernel first), the frame filter moving the
    # retained positions
    ("t128_13x13_c3584", wz.WZ_HAAR, wz.WZ_DB4, wz.WZ_BF16),
    ("frame_filter_T100", wz.WZ_HAAR, wz.WZ_BIOR44, wz.WZ_F32),
]


@pytest.mark.parametrize("name,tb,sb,out_dtype", CASES)
def test_condense_bases(name, tb, sb, out_dtype):
    wl, inp, out = _case(name, tb, sb)
    skip = _undecidable_frames(out, wl)
    print(f"[case] bases {name} temporal={NAMES[tb]} spatial={NAMES[sb]} T={wl.T} {wl.H}x{wl.W} C={wl.C} "
          f"Q={wl.Q} B={wl.B} out={out_dtype} undecidable frames={sorted(skip)}", flush=True)
    p = wz.problem_of(wl, out_dtype, temporal_basis=tb, spatial_basis=sb)
    X, q = wz.to_device(inp, DEV)
    tok, idx, b, o = wz.condense(p, X, q)
    torch.cuda.synchronize()
    tol = G.tol_for(wl.dtype) if out_dtype == wz.WZ_F32 else G.TOL_BF16_OUT
    _compare(wl, out, tok, idx, b, o, tol, skip)


@pytest.mark.parametrize("name,sb", [("tiny", wz.WZ_DB4), ("t64_14x14_c3584", wz.WZ_BIOR44),
                                     ("t128_13x13_c3584", wz.WZ_DB4), ("odd_3x5", wz.WZ_BIOR44),
                                     ("split_32x32_c200", wz.WZ_DB4)])
def test_stage_spatial_bases(name, sb):
    """wz_spatial_dwt_condense with a filter bank, fed the oracle's scores (as fp32) and offsets."""
    wl, inp, out = _case(name, wz.WZ_HAAR, sb)
    p = wz.problem_of(wl, wz.WZ_F32, spatial_basis=sb)
    X, _ = wz.to_device(inp, DEV)
    a32 = out["a"].astype(np.float32)
    a64 = a32.astype(np.float64)
    Xf = inp.X_f64()
    toks, idxs = [], []
    for t in range(wl.T):
        nt = int(out["budget"][t])
        if nt == 0:
            continue
        sel = oracle.select_tokens(a64[t], nt)
        Mt = oracle.saliency_map(a64[t]).reshape(wl.H, wl.W)
        mod = oracle.wavelet_spatial_modulator_bank(Xf[t], Mt, wl.lam, NAMES[sb]).reshape(wl.N, wl.C)
        toks.append(mod[sel])
        idxs.append(t * wl.N + sel)
    want_tok, want_idx = np.concatenate(toks), np.concatenate(idxs)
    offset = torch.from_numpy(out["offset"].astype(np.int32)).to(DEV)
    tok, idx = wz.spatial_dwt_condense(p, X, torch.from_numpy(a32.ravel()).to(DEV), offset)
    torch.cuda.synchronize()
    n = len(want_idx)
    assert np.array_equal(_np(idx)[:n], want_idx)
    assert G.within(_np(tok)[:n], want_tok, G.tol_for(wl.dtype))


@pytest.mark.parametrize("tb", [wz.WZ_DB4, wz.WZ_BIOR44])
@pytest.mark.parametrize("T", [1, 2, 3, 7, 64, 65, 300, 1025, 2048])
def test_stage_temporal_budget_bases(T, tb):
    """Random fp32 r and delta into wz_temporal_budget with a filter-bank allocator, J = 1..5."""
    rng = np.random.default_rng(1000 + T + 7 * tb)
    checked = 0
    for trial in range(6):
        N = int(rng.choice([1, 3, 196]))
        B = int(rng.integers(0, T * N + 1))
        levels = int(rng.integers(1, 6))
        tau = float(np.float32(rng.choice([0.0, 0.5])))
        r32 = rng.normal(0.05, 0.05, T).astype(np.float32)
        d32 = rng.uniform(0.0, 2.0, T).astype(np.float32)
        d32[0] = 0.0
        r64, d64 = r32.astype(np.float64), d32.astype(np.float64)
        kept = oracle.retained_frames(d64, tau)
        rt = oracle.wavelet_temporal_allocator_bank(r64[kept], oracle.temporal_gate(d64)[kept], levels, NAMES[tb])
        n, tr = oracle.allocate_budget_trace(rt, B, N)
        frac = np.sort(tr["q"] - np.floor(tr["q"]))[::-1]
        if 0 < tr["left"] < len(frac) and frac[tr["left"] - 1] - frac[tr["left"]] < 1e-9:
            continue  # a remainder tie within fp64 rounding: not a decidable comparison
        if np.any(np.abs(rt) < margins.M_R) and (tr["reactivated"] or tr["uniform"]):
            continue  # a weight sign within rounding decides the spread: not decidable either
        want = np.zeros(T, dtype=np.int64)
        want[kept] = n
        p = wz.Problem(T=T, H=1, W=N, C=8, Q=1, B=B, levels=levels, tau=tau, temporal_basis=tb)
        b, o, rr = wz.temporal_budget(p, torch.from_numpy(r32).to(DEV), torch.from_numpy(d32).to(DEV))
        torch.cuda.synchronize()
        assert np.array_equal(_np(b), want), (T, N, B, levels, tau)
        assert np.array_equal(_np(o), np.concatenate([[0], np.cumsum(want)]))
        want_rr = np.zeros(T)
        want_rr[kept] = rt
        assert G.rel_err(_np(rr), want_rr) <= 1e-6
        checked += 1
    assert checked > 0


@pytest.mark.parametrize("name,sb", [("split_32x32_c200", wz.WZ_DB4), ("split_27x27_c1152", wz.WZ_BIOR44)])
def test_split_form_matches_fused_kernel(name, sb):
    """bf16 inputs on a large grid: wz_condense runs the split form (the rows once per frame, then the
    contraction), wz_spatial_dwt_condense the fused kernel.  Both form the same bf16 operator rows and
    add each output's products in the same order (high then low part, 32-token step by step), so on the
    same scores and offsets their rows agree bit for bit."""
    wl, inp, _ = _case(name, wz.WZ_HAAR, sb)
    X, q = wz.to_device(inp, DEV)
    for out_dtype in (wz.WZ_BF16, wz.WZ_F32):
        p = wz.problem_of(wl, out_dtype, spatial_basis=sb)
        tok, idx, _, o = wz.condense(p, X, q)
        a, _, _ = wz.relevance(p, X, q)
        tok2, idx2 = wz.spatial_dwt_condense(p, X, a, o)
        torch.cuda.synchronize()
        n = int(o[-1].item())
        assert n > 0
        assert torch.equal(idx[:n], idx2[:n])
        assert torch.equal(tok[:n], tok2[:n])


@pytest.mark.parametrize("tb", [wz.WZ_BIOR44, wz.WZ_HAAR])
@pytest.mark.parametrize("name", ["tiny", "split_32x32_c200"])
def test_bases_batch_matches_single_calls(name, tb):
    """Two videos through wz_condense_batch with filter banks (the fused form, and the split form
    with bf16 inputs on a large grid; with the Haar temporal basis the budgets are computed in the
    modulator's first kernel): each bitwise equal to its single call."""
    wl, inp, _ = _case(name, tb, wz.WZ_DB4)
    p = wz.problem_of(wl, wz.WZ_F32 if wl.dtype == "f32" else wz.WZ_BF16, temporal_basis=tb,
                      spatial_basis=wz.WZ_DB4)
    X, q = wz.to_device(inp, DEV)
    X2, q2 = X.flip(0).contiguous(), q.flip(0).contiguous()
    tok, idx, b, o = wz.condense_batch(p, torch.stack([X, X2]), torch.stack([q, q2]))
    for v, (Xv, qv) in enumerate(((X, q), (X2, q2))):
        single = wz.condense(p, Xv, qv)
        torch.cuda.synchronize()
        for got, want in zip((tok[v], idx[v], b[v], o[v]), single):
            assert torch.equal(got, want)
