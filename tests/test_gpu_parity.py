"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Integer outputs (budgets, offsets, kept-token indices) must match bit-exactly;
floats within 2e-3 (bf16 inputs, fp32 accumulation) or 1e-5 (fp32 inputs),
relative error floored at 1e-3 of the tensor's largest magnitude.  Inputs are
the seeded workloads, whose decisions clear the tie margins, and small edge
cases.
"""
import numpy as np
import pytest
import torch

import gpu_util as G
import libutil
import oracle
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


def _run_case(wl, inp, out, out_dtype=wz.WZ_F32, check_stage1=True):
    p = wz.problem_of(wl, out_dtype)
    X, q = wz.to_device(inp, DEV)
    print(f"[case] {wl.name} T={wl.T} {wl.H}x{wl.W} C={wl.C} Q={wl.Q} B={wl.B} out={out_dtype}", flush=True)
    tol = G.tol_for(wl.dtype)
    if check_stage1:
        a, r, d = wz.relevance(p, X, q)
        torch.cuda.synchronize()
        assert G.within(_np(a), out["a"].ravel(), tol, f"{wl.name} a")
        assert G.within(_np(r), out["r"], tol, f"{wl.name} r")
        assert G.within(_np(d), out["delta"], tol, f"{wl.name} delta")
    tok, idx, b, o = wz.condense(p, X, q)
    torch.cuda.synchronize()
    n = int(out["offset"][-1])
    assert np.array_equal(_np(b), out["budget"])
    assert np.array_equal(_np(o), out["offset"])
    assert np.array_equal(_np(idx)[:n], out["index"])
    if out_dtype == wz.WZ_F32:
        assert G.within(_np(tok)[:n], out["tokens"], tol, f"{wl.name} tokens")
    else:
        assert G.within(_np(tok)[:n], out["tokens"], G.TOL_BF16_OUT, f"{wl.name} tokens (bf16 out)")
    return tok, idx, b, o


@pytest.mark.parametrize("name", synth.ORDER)
def test_workload_end_to_end(name):
    wl, inp, out = G.workload_case(name)
    assert G.check_margins(out, wl.N, wl.B, wl.tau) == []
    _run_case(wl, inp, out)


def test_benchmarked_launch_bf16_out_and_determinism():
    """The configuration the benchmark times (T=64 14x14 C=3584, bf16 out), twice: bitwise equal."""
    wl, inp, out = G.workload_case("t64_14x14_c3584")
    p = wz.problem_of(wl, wz.WZ_BF16)
    X, q = wz.to_device(inp, DEV)
    ws = wz.new_workspace(p, DEV)
    ws.fill_(0x5A)  # workspace contents on entry are ignored
    first = [t.clone() for t in wz.condense(p, X, q, ws=ws)]
    ws.fill_(0xA5)
    second = wz.condense(p, X, q, ws=ws)
    torch.cuda.synchronize()
    for x, y in zip(first, second):
        assert torch.equal(x.view(torch.int16) if x.dtype == torch.bfloat16 else x,
                           y.view(torch.int16) if y.dtype == torch.bfloat16 else y)
    tok, idx, b, _ = first
    assert np.array_equal(_np(b), out["budget"]) and np.array_equal(_np(idx), out["index"])
    assert G.within(_np(tok), out["tokens"], G.TOL_BF16_OUT)


@pytest.mark.parametrize("name", ["tiny", "t64_14x14_c3584"])
def test_relevance_pass_alone(name):
    """wz_relevance_pass writes the same per-token scores as wz_relevance (one slice: the pass completes them)."""
    wl, inp, out = G.workload_case(name)
    p = wz.problem_of(wl)
    X, q = wz.to_device(inp, DEV)
    ws = wz.new_workspace(p, DEV)
    a = torch.full((wl.T * wl.N,), float("nan"), dtype=torch.float32, device=DEV)
    wz.relevance_pass(p, X, q, a, ws)
    a_full, _, _ = wz.relevance(p, X, q)
    torch.cuda.synchronize()
    assert torch.equal(a, a_full)
    assert G.within(_np(a), out["a"].ravel(), G.tol_for(wl.dtype))


@pytest.mark.parametrize("name", ["tiny", "t64_14x14_c3584", "t128_13x13_c3584"])
def test_stage_temporal_budget(name):
    """wz_temporal_budget fed the oracle's r and delta (as fp32) vs the oracle's stage on the same values."""
    wl, inp, out = G.workload_case(name)
    p = wz.problem_of(wl)
    r32 = out["r"].astype(np.float32)
    d32 = out["delta"].astype(np.float32)
    r64, d64 = r32.astype(np.float64), d32.astype(np.float64)
    gamma = oracle.temporal_gate(d64)
    kept = oracle.retained_frames(d64, float(np.float32(wl.tau)))
    rt = oracle.wavelet_temporal_allocator(r64[kept], gamma[kept], wl.levels)
    n = oracle.allocate_budget(rt, wl.B, wl.N)
    want = np.zeros(wl.T, dtype=np.int64)
    want[kept] = n
    b, o, rr = wz.temporal_budget(p, torch.from_numpy(r32).to(DEV), torch.from_numpy(d32).to(DEV))
    torch.cuda.synchronize()
    assert np.array_equal(_np(b), want)
    assert np.array_equal(_np(o), np.concatenate([[0], np.cumsum(want)]))
    want_rr = np.zeros(wl.T)
    want_rr[kept] = rt
    assert G.rel_err(_np(rr), want_rr) <= 1e-6


def test_workspace_reuse_across_shapes():
    """One workspace serves calls of different shapes in turn."""
    big = G.workload_case("t64_14x14_c3584")
    small = G.workload_case("tiny")
    ws = wz.new_workspace(wz.problem_of(big[0]), DEV)
    for wl, inp, out in (big, small, big, small):
        X, q = wz.to_device(inp, DEV)
        tok, idx, b, o = wz.condense(wz.problem_of(wl), X, q, ws=ws)
        torch.cuda.synchronize()
        assert np.array_equal(_np(b), out["budget"]) and np.array_equal(_np(idx), out["index"])


@pytest.mark.parametrize("T", [1, 2, 3, 63, 64, 65, 100, 128, 129, 200, 255, 256, 257, 1023, 1024, 1025, 2048])
def test_stage_temporal_budget_random(T):
    """Random fp32 r and delta straight into wz_temporal_budget, up to the 2048-frame limit: one frame per
    lane of one wave up to 64 frames, four per lane up to 256 (with tau = 0.5 the frame filter drops frames,
    so the retained positions move), a workgroup above."""
    rng = np.random.default_rng(T)
    for trial in range(4):
        N = int(rng.choice([1, 3, 196]))
        B = int(rng.integers(0, T * N + 1))
        levels = int(rng.integers(1, 6))
        tau = float(np.float32(rng.choice([0.0, 0.5])))
        r32 = rng.normal(0.05, 0.05, T).astype(np.float32)
        d32 = rng.uniform(0.0, 2.0, T).astype(np.float32)
        d32[0] = 0.0
        r64, d64 = r32.astype(np.float64), d32.astype(np.float64)
        kept = oracle.retained_frames(d64, tau)
        rt = oracle.wavelet_temporal_allocator(r64[kept], oracle.temporal_gate(d64)[kept], levels)
        n, tr = oracle.allocate_budget_trace(rt, B, N)
        frac = np.sort(tr["q"] - np.floor(tr["q"]))[::-1]
        if 0 < tr["left"] < len(frac) and frac[tr["left"] - 1] - frac[tr["left"]] < 1e-9:
            continue  # a remainder tie within fp64 rounding: not a decidable comparison
        want = np.zeros(T, dtype=np.int64)
        want[kept] = n
        p = wz.Problem(T=T, H=1, W=N, C=8, Q=1, B=B, levels=levels, tau=tau)
        b, o, rr = wz.temporal_budget(p, torch.from_numpy(r32).to(DEV), torch.from_numpy(d32).to(DEV))
        torch.cuda.synchronize()
        assert np.array_equal(_np(b), want), (T, N, B, levels, tau)
        assert np.array_equal(_np(o), np.concatenate([[0], np.cumsum(want)]))
        want_rr = np.zeros(T)
        want_rr[kept] = rt
        assert G.rel_err(_np(rr), want_rr) <= 1e-6


@pytest.mark.parametrize("name,out_dtype", [("tiny", wz.WZ_F32), ("t64_14x14_c3584", wz.WZ_F32),
                                            ("t128_13x13_c3584", wz.WZ_BF16)])
def test_stage_spatial_condense(name, out_dtype):
    """wz_spatial_dwt_condense fed the oracle's scores (as fp32) and budgets vs the oracle's stage."""
    wl, inp, out = G.workload_case(name)
    p = wz.problem_of(wl, out_dtype)
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
        mod = oracle.wavelet_spatial_modulator(Xf[t], Mt, wl.lam).reshape(wl.N, wl.C)
        toks.append(mod[sel])
        idxs.append(t * wl.N + sel)
    want_tok, want_idx = np.concatenate(toks), np.concatenate(idxs)
    offset = torch.from_numpy(out["offset"].astype(np.int32)).to(DEV)
    tok, idx = wz.spatial_dwt_condense(p, X, torch.from_numpy(a32.ravel()).to(DEV), offset)
    torch.cuda.synchronize()
    n = len(want_idx)
    assert np.array_equal(_np(idx)[:n], want_idx)
    tol = G.TOL_BF16_OUT if out_dtype == wz.WZ_BF16 else G.tol_for(wl.dtype)
    assert G.within(_np(tok)[:n], want_tok, tol)


# ---------------------------------------------------------------------------
# Edge cases on small random inputs
# ---------------------------------------------------------------------------

def _random_case(seed, T, H, W, C, Q, B, dtype="bf16", levels=1, lam=1.5, tau=0.0, tweak=None):
    """A small random input (normal features, optional tweak) whose decisions clear the margins."""
    wl = synth.Workload(f"edge_T{T}_{H}x{W}_C{C}_Q{Q}_B{B}_{dtype}", T=T, H=H, W=W, C=C, Q=Q, dtype=dtype,
                        B=B, levels=levels, lam=lam, tau=tau)
    for s in range(seed, seed + 50):
        rng = np.random.default_rng(s)
        X = rng.standard_normal((T, H, W, C))
        q = rng.standard_normal((Q, C)) / np.sqrt(C)
        if tweak:
            X, q = tweak(X, q, rng)
        cast = (lambda v: synth.f32_to_bf16_bits(v.astype(np.float32))) if dtype == "bf16" else \
               (lambda v: v.astype(np.float32))
        inp = synth.Inputs(wl=wl, X=cast(X), query=cast(q))
        out = oracle.condense(inp.X_f64(), inp.query_f64(), B, levels, lam, float(np.float32(tau)))
        if not G.check_margins(out, wl.N, B, tau):
            return wl, inp, out
    raise AssertionError("no margin-clean seed for the edge case")


EDGE = {
    "odd_3x5": dict(T=5, H=3, W=5, C=64, Q=16, B=30),
    "row_1x7": dict(T=4, H=1, W=7, C=64, Q=16, B=9),
    "col_7x1": dict(T=4, H=7, W=1, C=64, Q=16, B=9),
    "single_token": dict(T=6, H=1, W=1, C=64, Q=16, B=4),
    "single_frame": dict(T=1, H=14, W=14, C=256, Q=32, B=37),
    "budget_zero": dict(T=8, H=4, W=4, C=64, Q=16, B=0),
    "budget_one": dict(T=8, H=4, W=4, C=64, Q=16, B=1),
    "budget_all": dict(T=8, H=4, W=4, C=64, Q=16, B=128),
    "ragged_channels": dict(T=6, H=6, W=6, C=40, Q=16, B=50),
    "min_channels": dict(T=6, H=6, W=6, C=8, Q=16, B=50),
    "ragged_query": dict(T=6, H=6, W=6, C=96, Q=17, B=50),
    "many_query": dict(T=6, H=6, W=6, C=96, Q=300, B=50),
    "small_query_bf16": dict(T=6, H=6, W=6, C=96, Q=5, B=50),
    "fp32_query32": dict(T=6, H=6, W=6, C=96, Q=32, B=50, dtype="f32"),
    "fp32_query1": dict(T=6, H=5, W=5, C=64, Q=1, B=40, dtype="f32"),
    "levels_4": dict(T=37, H=4, W=4, C=64, Q=16, B=150, levels=4),
    "odd_T_levels_2": dict(T=13, H=5, W=5, C=64, Q=16, B=90, levels=2),
    "frame_filter": dict(T=16, H=4, W=4, C=64, Q=16, B=100, tau=1.0),
    # the budgets inside the gather with four frames per lane, frames dropped
    # by the frame filter (their retained positions move) and several levels
    "frame_filter_T100": dict(T=100, H=4, W=4, C=64, Q=16, B=600, tau=1.0),
    "frame_filter_T200_levels_3": dict(T=200, H=3, W=3, C=32, Q=16, B=900, levels=3, tau=1.0),
    "lambda_zero": dict(T=4, H=4, W=4, C=64, Q=16, B=20, lam=0.0),
    "large_grid": dict(T=2, H=64, W=64, C=8, Q=16, B=3000),
    "many_frames": dict(T=512, H=2, W=2, C=16, Q=16, B=1900),
    "max_channels": dict(T=2, H=7, W=7, C=65536, Q=16, B=20),
    "max_query": dict(T=3, H=7, W=7, C=256, Q=1024, B=30),
    # four 16-column query tiles in the token-tiled pass: ragged query and
    # channels, a full 64-token tile, one-token frames, the most channels
    "query_47_ragged": dict(T=6, H=7, W=9, C=200, Q=47, B=60),
    "query_64_full_tile": dict(T=3, H=8, W=8, C=136, Q=64, B=40),
    "query_33_single_token": dict(T=5, H=1, W=1, C=72, Q=33, B=3),
    "query_64_max_channels": dict(T=2, H=7, W=7, C=65536, Q=64, B=20),
    # more than 64 query tokens in the token-tiled pass: passes of 32 columns
    # over each tile, the last one ragged; up to the most the pass takes
    "query_65_passes": dict(T=4, H=5, W=9, C=200, Q=65, B=40),
    "query_128_passes": dict(T=5, H=9, W=9, C=136, Q=128, B=60),
    "query_256_passes": dict(T=3, H=8, W=8, C=72, Q=256, B=30),
    "query_100_large_c": dict(T=2, H=7, W=7, C=16384, Q=100, B=20),
    # 17 to 32 query tokens (four-wave workgroups when the channel sums fit
    # LDS): one 64-channel chunk (three waves without a chunk), the largest
    # channel count whose sums fit, and one past it (eight waves)
    "query_20_one_chunk": dict(T=3, H=5, W=5, C=40, Q=20, B=20),
    "query_32_c8192": dict(T=2, H=7, W=7, C=8192, Q=32, B=20),
    "query_32_c8200": dict(T=2, H=7, W=7, C=8200, Q=32, B=20),
}


@pytest.mark.parametrize("case", sorted(EDGE))
def test_edge_case(case):
    wl, inp, out = _random_case(1000, **EDGE[case])
    for odt in (wz.WZ_F32, wz.WZ_BF16):
        _run_case(wl, inp, out, odt, check_stage1=(odt == wz.WZ_F32))


def _frame_filter_shortfall(X, q, rng):
    # every frame after the first repeats frame 0 up to a small change (delta ~ 0.05),
    # so tau = 0.3 drops them and B exceeds the single retained frame's tokens
    X[1:] = X[0] + 0.3 * rng.standard_normal(X[1:].shape)
    return X, q


def _zero_query_token(X, q, rng):
    q[1] = 0.0
    return X, q


def _zero_tokens(X, q, rng):
    X[0, 0, 0] = 0.0
    X[2, 1, 3] = 0.0
    return X, q


def _negative_relevance(X, q, rng):
    # the query points away from every frame's mean: every r_t < 0, all weights 0 -> uniform
    X = X + 3.0
    q = -np.abs(q) - 0.05
    return X, q


DEGENERATE = {
    "shortfall": dict(T=6, H=4, W=4, C=64, Q=16, B=40, tau=0.3, tweak=_frame_filter_shortfall),
    "zero_query_token": dict(T=5, H=4, W=4, C=64, Q=16, B=30, tweak=_zero_query_token),
    "zero_tokens": dict(T=5, H=4, W=4, C=64, Q=16, B=30, tweak=_zero_tokens),
    "negative_relevance": dict(T=6, H=4, W=4, C=64, Q=16, B=30, tweak=_negative_relevance),
}


@pytest.mark.parametrize("case", sorted(DEGENERATE))
def test_degenerate_case(case):
    wl, inp, out = _random_case(2000, **DEGENERATE[case])
    if case == "shortfall":
        assert out["retained"] == [0] and int(out["offset"][-1]) == wl.N < wl.B
    if case == "negative_relevance":
        assert np.all(out["r_tilde"] < 0)
    _run_case(wl, inp, out)


def test_identical_frames_exact():
    """Frames whose pooled features are exact multiples of one basis vector: delta = 0 exactly,
    every frame ties, and the budget is split evenly with leftovers to the earliest frames."""
    T, H, W, C, Q = 7, 4, 4, 8, 16
    X = np.zeros((T, H, W, C))
    X[..., 0] = 1.0
    rng = np.random.default_rng(5)
    q = rng.standard_normal((Q, C)) / np.sqrt(C)
    wl = synth.Workload("identical", T=T, H=H, W=W, C=C, Q=Q, dtype="bf16", B=20)
    inp = synth.Inputs(wl=wl, X=synth.f32_to_bf16_bits(X.astype(np.float32)),
                       query=synth.f32_to_bf16_bits(q.astype(np.float32)))
    out = oracle.condense(inp.X_f64(), inp.query_f64(), wl.B, 1, 1.5, 0.0)
    assert np.all(out["delta"] == 0.0) and out["budget"].tolist() == [3, 3, 3, 3, 3, 3, 2]
    _run_case(wl, inp, out)
