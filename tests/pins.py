"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Each `pin_*` function raises AssertionError when the oracle disagrees with a
closed form, an invariant, a hand-derived fixture or the pure-Python brute
force.  The pins run as ordinary tests, and again under planted mistakes
(test_oracle_mutations.py) to show that each plausible slip is caught.
"""
import itertools
import json
import math
import os

import numpy as np

import brute
import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _expr(s):
    """Evaluate a closed-form fixture expression (numbers, + - * / and sqrt only)."""
    allowed = set("0123456789.+-*/() sqrt")
    if not set(s) <= allowed:
        raise ValueError(f"unexpected characters in {s!r}")
    return float(eval(s, {"__builtins__": {}}, {"sqrt": math.sqrt}))


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# ---------------------------------------------------------------------------
# 1-D Haar and the temporal allocator (Eq. (9)-(11))
# ---------------------------------------------------------------------------

def pin_haar1d_hand_values():
    s2 = math.sqrt(2.0)
    A, D = oracle.haar_analysis(np.array([1.0, 3.0]))
    assert np.allclose(A, [4 / s2], rtol=0, atol=1e-15) and np.allclose(D, [-2 / s2], rtol=0, atol=1e-15)
    # odd length: [1, 2, 4] is extended to [1, 2, 4, 4]
    A, D = oracle.haar_analysis(np.array([1.0, 2.0, 4.0]))
    assert np.allclose(A, [3 / s2, 8 / s2], atol=1e-15) and np.allclose(D, [-1 / s2, 0.0], atol=1e-15)
    A, D = oracle.haar_analysis(np.array([5.0, 1.0, -2.0, 2.0]))
    assert np.allclose(A, [6 / s2, 0.0], atol=1e-15) and np.allclose(D, [4 / s2, -4 / s2], atol=1e-15)


def pin_haar1d_perfect_reconstruction():
    rng = np.random.default_rng(11)
    for n in range(1, 34):
        x = rng.standard_normal(n)
        A, D = oracle.haar_analysis(x)
        y = oracle.haar_synthesis(A, D, n)
        assert y.shape == (n,)
        assert np.max(np.abs(y - x)) <= 1e-12


def pin_haar1d_parseval():
    rng = np.random.default_rng(12)
    for n in range(2, 34, 2):
        x = rng.standard_normal(n)
        A, D = oracle.haar_analysis(x)
        assert abs(np.sum(x * x) - np.sum(A * A) - np.sum(D * D)) <= 1e-12 * np.sum(x * x)
    # odd length: energy of the extended signal
    x = rng.standard_normal(7)
    A, D = oracle.haar_analysis(x)
    xe = np.append(x, x[-1])
    assert abs(np.sum(xe * xe) - np.sum(A * A) - np.sum(D * D)) <= 1e-12 * np.sum(xe * xe)


def pin_haar1d_matrix_form():
    """Analysis equals the orthonormal Haar matrix applied to the signal."""
    n = 8
    Hm = np.zeros((n, n))
    for k in range(n // 2):
        Hm[k, 2 * k] = Hm[k, 2 * k + 1] = 1 / math.sqrt(2)
        Hm[n // 2 + k, 2 * k] = 1 / math.sqrt(2)
        Hm[n // 2 + k, 2 * k + 1] = -1 / math.sqrt(2)
    assert np.allclose(Hm @ Hm.T, np.eye(n), atol=1e-15)
    x = np.random.default_rng(13).standard_normal(n)
    A, D = oracle.haar_analysis(x)
    assert np.allclose(np.concatenate([A, D]), Hm @ x, atol=1e-14)


def pin_wta_special_cases():
    rng = np.random.default_rng(14)
    for L in range(1, 20):
        R = rng.standard_normal(L)
        for J in (1, 2, 3):
            # a fully open gate keeps every detail: perfect reconstruction
            assert np.max(np.abs(oracle.wavelet_temporal_allocator(R, np.ones(L), J) - R)) <= 1e-12
        # a closed gate at one level replaces each pair by its mean
        out = oracle.wavelet_temporal_allocator(R, np.zeros(L), 1)
        Re = np.append(R, R[-1]) if L % 2 else R
        means = np.repeat(0.5 * (Re[0::2] + Re[1::2]), 2)[:L]
        assert np.max(np.abs(out - means)) <= 1e-12
    # two closed levels on a length divisible by 4 give block means of 4
    R = rng.standard_normal(12)
    out = oracle.wavelet_temporal_allocator(R, np.zeros(12), 2)
    assert np.allclose(out, np.repeat(R.reshape(3, 4).mean(axis=1), 4), atol=1e-12)


def pin_wta_hand_gate():
    """J=1, R = (r0, r1), gate (g0, g1): r~0 = (r0+r1)/2 + g(r0-r1)/2 with g = (g0+g1)/2."""
    r0, r1, g0, g1 = 0.3, -0.1, 0.2, 0.6
    g = 0.5 * (g0 + g1)
    out = oracle.wavelet_temporal_allocator(np.array([r0, r1]), np.array([g0, g1]), 1)
    assert np.allclose(out, [(r0 + r1) / 2 + g * (r0 - r1) / 2, (r0 + r1) / 2 - g * (r0 - r1) / 2], atol=1e-15)
    # J=2 on four samples with gates (1,0,0,1): level-1 details scaled by (1/2, 1/2), level 2 by 1/2
    R = np.array([1.0, 2.0, 4.0, 8.0])
    out = oracle.wavelet_temporal_allocator(R, np.array([1.0, 0.0, 0.0, 1.0]), 2)
    pair = np.array([1.5, 6.0])                    # level-1 approximations / sqrt2
    top = pair.mean() + 0.5 * (pair - pair.mean())  # level-2 detail halved
    expect = np.array([top[0] - 0.25, top[0] + 0.25, top[1] - 1.0, top[1] + 1.0])
    assert np.allclose(out, expect, atol=1e-12)


# ---------------------------------------------------------------------------
# 2-D Haar and the spatial modulator (Eq. (12)-(15))
# ---------------------------------------------------------------------------

def pin_haar2d_explicit_butterflies():
    rng = np.random.default_rng(21)
    F = rng.standard_normal((4, 6, 3))
    LL, LH, HL, HH = oracle.haar_analysis_2d(F)
    p00, p01, p10, p11 = F[0::2, 0::2], F[0::2, 1::2], F[1::2, 0::2], F[1::2, 1::2]
    assert np.allclose(LL, (p00 + p01 + p10 + p11) / 2, atol=1e-14)
    assert np.allclose(LH, (p00 - p01 + p10 - p11) / 2, atol=1e-14)
    assert np.allclose(HL, (p00 + p01 - p10 - p11) / 2, atol=1e-14)
    assert np.allclose(HH, (p00 - p01 - p10 + p11) / 2, atol=1e-14)


def pin_haar2d_reconstruction_and_parseval():
    rng = np.random.default_rng(22)
    for H, W in [(2, 2), (3, 3), (4, 7), (13, 13), (14, 14), (1, 5), (5, 1)]:
        F = rng.standard_normal((H, W, 2))
        bands = oracle.haar_analysis_2d(F)
        assert np.max(np.abs(oracle.haar_synthesis_2d(*bands, H, W) - F)) <= 1e-12
        Fe = np.concatenate([F, F[-1:]], axis=0) if H % 2 else F
        Fe = np.concatenate([Fe, Fe[:, -1:]], axis=1) if W % 2 else Fe
        energy = sum(np.sum(b * b) for b in bands)
        assert abs(energy - np.sum(Fe * Fe)) <= 1e-12 * np.sum(Fe * Fe)


def pin_wsm_closed_form():
    """Gating the three detail bands by g gives mu_b + g (x - mu_b) on each padded 2x2 block."""
    rng = np.random.default_rng(23)
    for H, W in [(2, 2), (3, 5), (14, 14), (13, 13)]:
        F = rng.standard_normal((H, W, 3))
        M = rng.random((H, W))
        lam = 1.5
        out = oracle.wavelet_spatial_modulator(F, M, lam)
        for h in range(H):
            for w in range(W):
                rows = [h - h % 2, min(h - h % 2 + 1, H - 1)]
                cols = [w - w % 2, min(w - w % 2 + 1, W - 1)]
                mu = sum(F[r, c] for r in rows for c in cols) / 4
                g = lam * sum(M[r, c] for r in rows for c in cols) / 4
                assert np.allclose(out[h, w], mu + g * (F[h, w] - mu), atol=1e-12)


def pin_wsm_unit_and_zero_gate():
    rng = np.random.default_rng(24)
    F = rng.standard_normal((5, 7, 4))
    # lambda * mean(M) = 1 everywhere: identity
    assert np.allclose(oracle.wavelet_spatial_modulator(F, np.full((5, 7), 2 / 3), 1.5), F, atol=1e-12)
    # lambda = 0: every token becomes its (padded) block mean
    out = oracle.wavelet_spatial_modulator(F, rng.random((5, 7)), 0.0)
    assert np.allclose(out[0, 0], F[0:2, 0:2].mean(axis=(0, 1)), atol=1e-12)
    assert np.allclose(out[4, 6], F[4, 6], atol=1e-12)            # corner block is one token repeated
    assert np.allclose(out[4, 2], F[4, 2:4].mean(axis=0), atol=1e-12)


# ---------------------------------------------------------------------------
# Scores and the visual change estimator (Sec. 3.2.1, Eq. (7), Eq. (8))
# ---------------------------------------------------------------------------

def pin_cosine_cases():
    v = np.array([[1.0, 2.0, -1.0]])
    X = np.stack([np.stack([np.tile(v, (2, 1))] * 2)] * 3)   # three identical frames
    d = oracle.visual_change(oracle.pooled_features(X))
    assert np.allclose(d, 0.0, atol=1e-15)
    ortho = np.array([[1.0, 0.0]]), np.array([[0.0, 3.0]])
    anti = np.array([[1.0, -2.0]]), np.array([[-2.0, 4.0]])
    assert abs(oracle.visual_change(np.concatenate(ortho))[1] - 1.0) <= 1e-15
    assert abs(oracle.visual_change(np.concatenate(anti))[1] - 2.0) <= 1e-15
    assert oracle.visual_change(np.array([[0.0, 0.0], [1.0, 2.0]]))[1] == 1.0   # zero vector: cos = 0
    assert np.allclose(oracle.cosine_matrix(np.array([[2.0, 0.0]]), np.array([[0.0, 0.0], [5.0, 0.0]])), [[0.0, 1.0]])


def pin_scores_scale_invariance_and_range():
    rng = np.random.default_rng(31)
    X = rng.standard_normal((3, 4, 5, 6))
    q = rng.standard_normal((3, 6))
    a = oracle.token_saliency(X, q)
    assert a.shape == (3, 20) and np.all(a <= 1 + 1e-15) and np.all(a >= -1 - 1e-15)
    scale = rng.random((3, 4, 5, 1)) + 0.5
    assert np.allclose(oracle.token_saliency(X * scale, q * 7.0), a, atol=1e-14)
    # a token equal to a query token scores 1
    X2 = X.copy()
    X2[1, 2, 3] = 4.0 * q[2]
    assert abs(oracle.token_saliency(X2, q)[1, 2 * 5 + 3] - 1.0) <= 1e-14
    # max over query tokens, brute loop
    for t, n in [(0, 0), (2, 19)]:
        x = X[t].reshape(20, 6)[n]
        best = max(float(x @ qj) / (np.linalg.norm(x) * np.linalg.norm(qj)) for qj in q)
        assert abs(a[t, n] - best) <= 1e-14
    # relevance uses the pooled mean; scaling tokens of a frame uniformly leaves r unchanged
    r = oracle.frame_relevance(oracle.pooled_features(X), q)
    r2 = oracle.frame_relevance(oracle.pooled_features(X * 3.0), q)
    assert np.allclose(r, r2, atol=1e-14)


def pin_minmax_maps():
    a = np.array([0.2, -0.4, 0.8, 0.8])
    M = oracle.saliency_map(a)
    assert np.allclose(M, [0.5, 0.0, 1.0, 1.0]) and oracle.saliency_map(np.full(4, 0.3)).tolist() == [0.0] * 4
    g = oracle.temporal_gate(np.array([0.0, 0.5, 0.25, 1.0]))
    assert np.allclose(g, [0.0, 0.5, 0.25, 1.0])
    assert oracle.retained_frames(np.array([0.0, 0.1, 0.3, 0.05, 0.3]), 0.3) == [0, 2, 4]


# ---------------------------------------------------------------------------
# Budgets (Eq. (16) under Eq. (5))
# ---------------------------------------------------------------------------

def pin_budget_hand_cases():
    assert oracle.allocate_budget(np.array([10.0, 1.0, 1.0]), 6, 4).tolist() == [4, 1, 1]    # cap then re-apportion
    assert oracle.allocate_budget(np.array([0.3, 0.2, 0.5]), 7, 10).tolist() == [2, 1, 4]    # 2.1, 1.4, 3.5
    assert oracle.allocate_budget(np.array([1.0, 1.0, 1.0]), 4, 10).tolist() == [2, 1, 1]    # ties -> smaller index
    assert oracle.allocate_budget(np.array([-1.0, -0.5, 0.0]), 5, 10).tolist() == [2, 2, 1]  # all weights zero: uniform
    assert oracle.allocate_budget(np.array([0.5, -1.0, 0.5]), 4, 10).tolist() == [2, 0, 2]   # negative relevance gets 0
    assert oracle.allocate_budget(np.array([0.5, 0.1]), 30, 10).tolist() == [10, 10]          # shortfall: all full
    assert oracle.allocate_budget(np.array([5.0, 0.0, 0.0]), 6, 4).tolist() == [4, 1, 1]      # full, then spread evenly
    assert oracle.allocate_budget(np.array([0.2, 0.7]), 0, 10).tolist() == [0, 0]


def pin_budget_invariants(cases=300, seed=41):
    rng = np.random.default_rng(seed)
    for _ in range(cases):
        L = int(rng.integers(1, 12))
        N = int(rng.integers(1, 30))
        B = int(rng.integers(0, L * N + 5))
        w = rng.standard_normal(L) * rng.choice([1e-3, 1.0, 100.0])
        n = oracle.allocate_budget(w, B, N)
        assert n.sum() == min(B, L * N)
        assert np.all(n >= 0) and np.all(n <= N)
        pos = np.maximum(w, 0)
        if B < L * N and pos.sum() > 0:
            q = B * pos / pos.sum()
            if np.all(q < N):
                assert np.all((n == np.floor(q)) | (n == np.ceil(q)))
                assert np.all(n[pos == 0] == 0)


def pin_budget_least_squares_brute():
    """Without caps, largest remainders minimise sum (n - q)^2 over integer vectors with sum B."""
    rng = np.random.default_rng(42)
    for _ in range(60):
        L = int(rng.integers(1, 5))
        N = 8
        B = int(rng.integers(0, 9))
        w = rng.random(L) + 0.05
        q = B * w / w.sum()
        if np.any(q >= N):
            continue
        n = oracle.allocate_budget(w, B, N)
        best = min(sum((c - qq) ** 2 for c, qq in zip(v, q))
                   for v in itertools.product(range(N + 1), repeat=L) if sum(v) == B)
        assert abs(sum((c - qq) ** 2 for c, qq in zip(n, q)) - best) <= 1e-12


def pin_budget_matches_brute():
    rng = np.random.default_rng(43)
    for _ in range(200):
        L = int(rng.integers(1, 7))
        N = int(rng.integers(1, 9))
        B = int(rng.integers(0, L * N + 3))
        w = rng.standard_normal(L)
        assert oracle.allocate_budget(w, B, N).tolist() == brute._apportion(list(w), B, N)


# ---------------------------------------------------------------------------
# Selection and end to end
# ---------------------------------------------------------------------------

def pin_selection_brute():
    rng = np.random.default_rng(51)
    for _ in range(100):
        N = int(rng.integers(1, 12))
        a = np.round(rng.standard_normal(N), 1)          # rounded: many exact ties
        n = int(rng.integers(0, N + 1))
        expect = sorted(sorted(range(N), key=lambda i: (-a[i], i))[:n])
        assert oracle.select_tokens(a, n).tolist() == expect


def _check_golden(fix, out):
    exp = fix["expect"]
    for key in ("a", "r", "delta", "gamma", "r_tilde"):
        if key in exp:
            want = np.array([[_expr(e) for e in row] for row in exp[key]] if isinstance(exp[key][0], list)
                            else [_expr(e) for e in exp[key]])
            assert np.allclose(np.asarray(out[key]), want, rtol=0, atol=1e-14), key
    assert list(out["budget"]) == exp["budget"]
    assert list(out["index"]) == exp["index"]
    want = np.array([[_expr(e) for e in row] for row in exp["tokens"]])
    assert np.allclose(np.asarray(out["tokens"]), want, rtol=0, atol=1e-14)


def pin_golden_hand_cases():
    for name in ("hand_2frame_2x2.json", "hand_1frame_3x3.json"):
        fix = _load(name)
        X, q = np.array(fix["X"], dtype=float), np.array(fix["query"], dtype=float)
        out = oracle.condense(X, q, fix["B"], fix["levels"], fix["lam"], fix["tau"])
        _check_golden(fix, out)
        _check_golden(fix, brute.condense(fix["X"], fix["query"], fix["B"], fix["levels"], fix["lam"], fix["tau"]))
        if "modulated_frame" in fix["expect"]:
            Mt = oracle.saliency_map(out["a"][0]).reshape(3, 3)
            mod = oracle.wavelet_spatial_modulator(X[0], Mt, fix["lam"])[:, :, 0]
            want = np.array([[_expr(e) for e in row] for row in fix["expect"]["modulated_frame"]])
            assert np.allclose(mod, want, atol=1e-14)


def pin_end_to_end_brute(cases=40, seed=61):
    rng = np.random.default_rng(seed)
    for _ in range(cases):
        T, H, W = (int(v) for v in rng.integers(1, 5, size=3))
        C, Q = int(rng.integers(1, 4)), int(rng.integers(1, 3))
        X = rng.standard_normal((T, H, W, C))
        q = rng.standard_normal((Q, C))
        B = int(rng.integers(0, T * H * W + 2))
        J = int(rng.integers(1, 3))
        tau = float(rng.choice([0.0, 0.4]))
        o = oracle.condense(X, q, B, J, 1.5, tau)
        b = brute.condense(X.tolist(), q.tolist(), B, J, 1.5, tau)
        assert list(o["budget"]) == b["budget"]
        assert list(o["index"]) == b["index"]
        assert np.allclose(o["tokens"], np.array(b["tokens"]).reshape(o["tokens"].shape), atol=1e-12)
        assert np.allclose(o["r_tilde"], b["r_tilde"], atol=1e-12)


def pin_interp_identity_and_grid():
    """Psi at n = H*W is the identity; the grid keeps every row occupied and the aspect ratio."""
    for H, W in ((14, 14), (3, 5), (7, 1), (13, 13)):
        rng = np.random.default_rng(H * 31 + W)
        X = rng.standard_normal((H, W, 2))
        out, near = oracle.budget_guided_interpolation(X, H * W)
        assert np.array_equal(out, X.reshape(H * W, 2)) and np.array_equal(near, np.arange(H * W))
        for n in range(1, H * W + 1):
            h, w = oracle.interpolation_grid(n, H, W)
            h0 = min(H, max(1, int(np.floor(np.sqrt(n * H / W) + 0.5))))
            assert w == min(W, -(-n // h0)) and h * w >= n > (h - 1) * w


def pin_interp_affine_exact():
    """Bilinear interpolation at half-pixel centres reproduces an affine map exactly
    (coordinates clamped at 0); the index is the nearest token, halves up."""
    H, W = 13, 11
    yy, xx = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
    X = (0.75 * yy - 1.25 * xx + 0.5)[:, :, None]
    for n in (1, 2, 5, 17, 40, 100, 142):
        out, near = oracle.budget_guided_interpolation(X, n)
        h, w = oracle.interpolation_grid(n, H, W)
        for k in range(n):
            i, j = divmod(k, w)
            sy, sx = max(0.0, (i + 0.5) * H / h - 0.5), max(0.0, (j + 0.5) * W / w - 0.5)
            assert abs(out[k, 0] - (0.75 * sy - 1.25 * sx + 0.5)) < 1e-12
            ny, nx = min(H - 1, math.floor((i + 0.5) * H / h)), min(W - 1, math.floor((j + 0.5) * W / w))
            assert near[k] == ny * W + nx


def _two_level_closed_form(F, M, lam):
    """x~ = mu2 + g2 (mu1 - mu2) + g1 (x - mu1), written out with explicit index clamping:
    mu1 / g1 over the token's 2x2 block, mu2 / g2 over the 2x2 level-1 cells of its
    level-2 block (the last row / column repeated at each level)."""
    H, W = M.shape
    Hb, Wb = (H + 1) // 2, (W + 1) // 2

    def cell(A, bi, bj):  # mean over level-1 cell (bi, bj) of a token map
        return 0.25 * sum(A[min(2 * bi + a, H - 1), min(2 * bj + b, W - 1)] for a in (0, 1) for b in (0, 1))

    def block2(A, ci, cj):  # mean over the level-1 cells of level-2 block (ci, cj)
        return 0.25 * sum(cell(A, min(2 * ci + a, Hb - 1), min(2 * cj + b, Wb - 1)) for a in (0, 1) for b in (0, 1))

    out = np.zeros_like(F)
    for h in range(H):
        for w in range(W):
            bi, bj = h // 2, w // 2
            mu1, mu2 = cell(F, bi, bj), block2(F, bi // 2, bj // 2)
            g1, g2 = lam * cell(M, bi, bj), lam * block2(M, bi // 2, bj // 2)
            out[h, w] = mu2 + g2 * (mu1 - mu2) + g1 * (F[h, w] - mu1)
    return out


def pin_wsm_two_levels():
    """The two-level spatial modulator: its closed form on random maps, the identity under a unit gate and the
    level-2 approximation under a zero gate (odd and even grids)."""
    rng = np.random.default_rng(5)
    for H, W in ((14, 14), (13, 13), (5, 7), (2, 3), (1, 1)):
        F = rng.standard_normal((H, W, 3))
        M = rng.random((H, W))
        got = oracle.wavelet_spatial_modulator(F, M, 1.5, 2)
        assert np.abs(got - _two_level_closed_form(F, M, 1.5)).max() < 1e-12
        assert np.abs(oracle.wavelet_spatial_modulator(F, np.full((H, W), 2.0), 0.5, 2) - F).max() < 1e-12
        flat = oracle.wavelet_spatial_modulator(F, np.zeros((H, W)), 1.5, 2)
        assert np.abs(flat - _two_level_closed_form(F, np.zeros((H, W)), 1.5)).max() < 1e-12


# ---------------------------------------------------------------------------
# Longer wavelet bases: db4 and bior4.4 (Sec. 3.2.3, Sec. 4.3)
# ---------------------------------------------------------------------------

BANKS = ("haar", "db4", "bior4.4")


def pin_wavelet_taps_published():
    """The constructed low-pass filters equal the published tables (tests/golden/wavelet_taps.json)."""
    fix = _load("wavelet_taps.json")
    h = oracle.daubechies_lowpass(4)
    assert np.abs(h - np.array(fix["db4_lowpass"]["values"])).max() < 1e-12
    ana, syn = oracle.cdf_lowpasses()
    a = np.array(fix["cdf97_analysis_lowpass"]["center_out"]) * math.sqrt(2.0)
    g = np.array(fix["cdf97_synthesis_lowpass"]["center_out"]) / math.sqrt(2.0)
    assert np.abs(ana - np.concatenate([a[:0:-1], a])).max() < 1e-12
    assert np.abs(syn - np.concatenate([g[:0:-1], g])).max() < 1e-12
    dec_lo, _, rec_lo, _ = oracle.filter_bank("db4")
    assert np.array_equal(rec_lo, h) and np.array_equal(dec_lo, h[::-1])


def pin_wavelet_filter_algebra():
    """db4: orthonormal (sum_k h_k h_(k+2m) = delta_m), sum sqrt 2; bior4.4: symmetric low-passes,
    biorthogonal (sum_k dec_lo[k] rec_lo[k + 2m] reversed-aligned = delta_m); every high-pass of the
    longer bases kills polynomials of degree < 4 (four vanishing moments), Haar's constants."""
    for basis, moments in (("haar", 1), ("db4", 4), ("bior4.4", 4)):
        dec_lo, dec_hi, rec_lo, rec_hi = oracle.filter_bank(basis)
        F = len(dec_lo)
        assert F % 2 == 0 and len(dec_hi) == len(rec_lo) == len(rec_hi) == F
        assert abs(dec_lo.sum() - math.sqrt(2.0)) < 1e-13 and abs(rec_lo.sum() - math.sqrt(2.0)) < 1e-13
        k = np.arange(F, dtype=np.float64)
        for p in range(moments):
            assert abs(np.sum(dec_hi * k ** p)) < 1e-10 * F ** p, (basis, p)
            assert abs(np.sum(rec_hi * k ** p)) < 1e-10 * F ** p, (basis, p)
        # biorthogonality of the analysis and synthesis low-passes: with the
        # analysis filter reversed, sum_k rev(dec_lo)[k] rec_lo[k + 2m] = delta_m
        rd = dec_lo[::-1]
        for m in range(-(F // 2) + 1, F // 2):
            v = sum(rd[i] * rec_lo[i + 2 * m] for i in range(F) if 0 <= i + 2 * m < F)
            assert abs(v - (1.0 if m == 0 else 0.0)) < 1e-12, (basis, m)
    h = oracle.daubechies_lowpass(4)
    for m in range(4):
        assert abs(sum(h[i] * h[i + 2 * m] for i in range(8 - 2 * m)) - (1.0 if m == 0 else 0.0)) < 1e-13
    ana, syn = oracle.cdf_lowpasses()
    assert np.abs(ana - ana[::-1]).max() < 1e-14 and np.abs(syn - syn[::-1]).max() < 1e-14


def pin_dwt_bank_perfect_reconstruction():
    """dwt_step then idwt_step is the identity for every basis, every length 1..40, along any axis;
    the 2-D step likewise on odd and even grids."""
    rng = np.random.default_rng(71)
    for basis in BANKS:
        bank = oracle.filter_bank(basis)
        for L in range(1, 41):
            x = rng.standard_normal((L, 2))
            a, d = oracle.dwt_step(x, bank)
            assert a.shape[0] == (L + len(bank[0]) - 1) // 2
            assert np.abs(oracle.idwt_step(a, d, bank, L) - x).max() < 1e-12, (basis, L)
        y = rng.standard_normal((3, 9, 2))
        a, d = oracle.dwt_step(y, bank, axis=1)
        assert np.abs(oracle.idwt_step(a, d, bank, 9, axis=1) - y).max() < 1e-12
        for H, W in ((14, 14), (13, 13), (27, 27), (1, 5), (6, 3)):
            F = rng.standard_normal((H, W, 3))
            assert np.abs(oracle.idwt2_step(*oracle.dwt2_step(F, bank), bank, H, W) - F).max() < 1e-12


def pin_dwt_bank_matches_brute():
    """The vectorised steps equal the scalar brute force of tests/brute.py (explicit mirrored list,
    scatter-form synthesis) on tiny signals of every basis."""
    rng = np.random.default_rng(72)
    for basis in BANKS:
        dec_lo, dec_hi, rec_lo, rec_hi = (list(map(float, v)) for v in oracle.filter_bank(basis))
        bank = oracle.filter_bank(basis)
        for L in (1, 2, 3, 4, 7, 10, 14):
            x = rng.standard_normal(L)
            a, d = oracle.dwt_step(x, bank)
            ba, bd = brute.dwt_bank(list(x), dec_lo, dec_hi)
            assert np.abs(a - ba).max() < 1e-13 and np.abs(d - bd).max() < 1e-13
            g = rng.standard_normal((2, len(ba)))
            assert np.abs(oracle.idwt_step(g[0], g[1], bank, L)
                          - brute.idwt_bank(list(g[0]), list(g[1]), rec_lo, rec_hi, L)).max() < 1e-13


def pin_dwt_bank_haar_is_haar():
    """With the Haar bank the general steps are the Haar steps (odd lengths too), in 1-D and 2-D."""
    rng = np.random.default_rng(73)
    bank = oracle.filter_bank("haar")
    for L in range(1, 12):
        x = rng.standard_normal((L, 2))
        A, D = oracle.haar_analysis(x)
        a, d = oracle.dwt_step(x, bank)
        assert np.abs(A - a).max() < 1e-15 and np.abs(D - d).max() < 1e-15
        assert np.abs(oracle.idwt_step(a, d, bank, L) - oracle.haar_synthesis(A, D, L)).max() < 1e-15
    F = rng.standard_normal((5, 6, 2))
    for u, v in zip(oracle.dwt2_step(F, bank), oracle.haar_analysis_2d(F)):
        assert np.abs(u - v).max() < 1e-15


def pin_dwt_bank_periodic_parseval():
    """Periodised, the orthonormal bases keep energy (sum a^2 + sum d^2 = sum x^2) and are invertible by
    their transpose; the biorthogonal bior4.4 does not keep energy (its rows are not orthonormal)."""
    rng = np.random.default_rng(74)
    for basis in ("haar", "db4"):
        bank = oracle.filter_bank(basis)
        for L in (8, 14, 16, 30):
            x = rng.standard_normal(L)
            a, d = oracle.dwt_step(x, bank, mode="periodization")
            assert abs(np.sum(a * a) + np.sum(d * d) - np.sum(x * x)) < 1e-12 * np.sum(x * x), (basis, L)
            Wm = np.stack([np.concatenate(oracle.dwt_step(e, bank, mode="periodization")) for e in np.eye(L)], 1)
            assert np.abs(Wm @ Wm.T - np.eye(L)).max() < 1e-12
    x = rng.standard_normal(16)
    a, d = oracle.dwt_step(x, oracle.filter_bank("bior4.4"), mode="periodization")
    assert abs(np.sum(a * a) + np.sum(d * d) - np.sum(x * x)) > 1e-6 * np.sum(x * x)


def pin_dwt_bank_constants_and_cubics():
    """A constant signal has no detail anywhere (the symmetric extension of a constant is constant) and
    approximation sqrt 2 times it; the details of a cubic vanish wherever the analysis filter does not reach
    past the ends (four vanishing moments of db4 and bior4.4)."""
    for basis in BANKS:
        bank = oracle.filter_bank(basis)
        F = len(bank[0])
        for L in (1, 5, 14):
            a, d = oracle.dwt_step(np.full(L, 3.0), bank)
            assert np.abs(d).max() < 1e-13 and np.abs(a - 3.0 * math.sqrt(2.0)).max() < 1e-12
        if basis == "haar":
            continue
        L = 40
        t = np.arange(L, dtype=np.float64)
        x = 0.5 * t ** 3 - 4.0 * t ** 2 + t - 7.0
        _, d = oracle.dwt_step(x, bank)
        # d[k] reads x~[2k + 1 - j], j < F: inside [0, L) for F - 1 <= 2k + 1 <= L - 1
        inner = [k for k in range(len(d)) if 2 * k + 1 - (F - 1) >= 0 and 2 * k + 1 <= L - 1]
        assert len(inner) > 5
        assert np.abs(d[inner]).max() < 1e-8 * np.abs(x).max(), basis
        assert np.abs(d).max() > 1e-3  # the ends do feel the extension


def pin_adaptive_average_torch():
    """`adaptive_average` equals torch's adaptive average pooling (an independent implementation), 1-D and
    2-D, for shrinking and equal sizes; pairs of an even length are pair averages."""
    import torch
    rng = np.random.default_rng(75)
    for L in range(1, 30):
        for n in range(1, L + 1):
            v = rng.standard_normal(L)
            want = torch.nn.functional.adaptive_avg_pool1d(torch.tensor(v)[None, None], n)[0, 0].numpy()
            assert np.abs(oracle.adaptive_average(v, n) - want).max() < 1e-12, (L, n)
    M = rng.random((14, 13))
    want = torch.nn.functional.adaptive_avg_pool2d(torch.tensor(M)[None, None], (10, 10))[0, 0].numpy()
    got = oracle.adaptive_average(oracle.adaptive_average(M, 10, axis=0), 10, axis=1)
    assert np.abs(got - want).max() < 1e-12
    g = rng.standard_normal(12)
    assert np.abs(oracle.adaptive_average(g, 6) - oracle.pair_average(g)).max() < 1e-15


def pin_wta_bank_cases():
    """Temporal allocator with a filter bank: gate 1 rebuilds r exactly (every basis, J = 1..3, odd lengths);
    with the Haar bank and lengths divisible by 2^J it is the Haar allocator; gate 0 keeps only the coarsest
    approximation, which for a constant sequence is the sequence itself."""
    rng = np.random.default_rng(76)
    for basis in ("db4", "bior4.4"):
        for J in (1, 2, 3):
            for L in (1, 7, 16, 33, 64):
                r = rng.standard_normal(L)
                assert np.abs(oracle.wavelet_temporal_allocator_bank(r, np.ones(L), J, basis) - r).max() < 1e-12
            c = np.full(21, -0.7)
            assert np.abs(oracle.wavelet_temporal_allocator_bank(c, np.zeros(21), J, basis) - c).max() < 1e-12
    for J in (1, 2, 3):
        L = 8 * 2 ** J
        r, g = rng.standard_normal(L), rng.random(L)
        want = oracle.wavelet_temporal_allocator(r, g, J)
        assert np.abs(oracle.wavelet_temporal_allocator_bank(r, g, J, "haar") - want).max() < 1e-13


def pin_wsm_bank_cases():
    """Spatial modulator with a filter bank: a unit gate rebuilds the frame (odd and even grids); with the
    Haar bank on even grids it is the Haar modulator; the result is affine in lambda with the approximation-only
    frame at lambda = 0; a constant frame is left unchanged by any gate."""
    rng = np.random.default_rng(77)
    for basis in ("db4", "bior4.4"):
        for H, W in ((14, 14), (13, 13), (27, 27), (3, 8)):
            F = rng.standard_normal((H, W, 2))
            M = rng.random((H, W))
            assert np.abs(oracle.wavelet_spatial_modulator_bank(F, np.full((H, W), 0.5), 2.0, basis) - F).max() < 1e-12
            x0 = oracle.wavelet_spatial_modulator_bank(F, M, 0.0, basis)
            x1 = oracle.wavelet_spatial_modulator_bank(F, M, 1.0, basis)
            x15 = oracle.wavelet_spatial_modulator_bank(F, M, 1.5, basis)
            assert np.abs(x15 - (x0 + 1.5 * (x1 - x0))).max() < 1e-12
            C = np.full((H, W, 2), 1.25)
            assert np.abs(oracle.wavelet_spatial_modulator_bank(C, M, 1.5, basis) - C).max() < 1e-12
    for H, W in ((14, 14), (4, 6)):
        F = rng.standard_normal((H, W, 3))
        M = rng.random((H, W))
        want = oracle.wavelet_spatial_modulator(F, M, 1.5)
        assert np.abs(oracle.wavelet_spatial_modulator_bank(F, M, 1.5, "haar") - want).max() < 1e-13


ALL_PINS = [v for k, v in sorted(globals().items()) if k.startswith("pin_")]
