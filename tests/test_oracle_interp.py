"""Pins of the oracle's budget-guided interpolation (Psi of Eq. (17), under the
grid reading stated in the oracle's header): grid invariants, the identity at
n = H*W, exactness on affine maps, and agreement with two independent bilinear
routines (torch's interpolate with half-pixel centres, scipy's map_coordinates)."""
import numpy as np
import pytest
import scipy.ndimage
import torch

import oracle

SHAPES = [(14, 14), (13, 13), (8, 8), (3, 5), (1, 7), (7, 1), (27, 27), (5, 9)]


def _pos(i, L, l):
    return max(0.0, (i + 0.5) * L / l - 0.5)


@pytest.mark.parametrize("H,W", SHAPES)
def test_grid_invariants(H, W):
    for n in range(1, H * W + 1):
        h, w = oracle.interpolation_grid(n, H, W)
        assert 1 <= h <= H and 1 <= w <= W
        assert h * w >= n and (h - 1) * w < n  # every row holds a cell
        # h0 is the integer nearest sqrt(n H / W) (halves up), within [1, H]
        h0 = min(H, max(1, int(np.floor(np.sqrt(n * H / W) + 0.5))))
        assert w == min(W, -(-n // h0))


@pytest.mark.parametrize("H,W", SHAPES)
def test_identity_at_full_budget(H, W):
    rng = np.random.default_rng(H * 100 + W)
    X = rng.standard_normal((H, W, 3))
    out, near = oracle.budget_guided_interpolation(X, H * W)
    assert np.array_equal(out, X.reshape(H * W, 3))
    assert np.array_equal(near, np.arange(H * W))


@pytest.mark.parametrize("H,W", SHAPES)
def test_affine_maps_are_exact(H, W):
    """Bilinear interpolation reproduces an affine map at the (clamped) sample point."""
    a, b, c = 0.75, -1.25, 0.5
    yy, xx = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
    X = (a * yy + b * xx + c)[:, :, None]
    for n in sorted({1, 2, 3, 7, (H * W) // 3 + 1, H * W - 1, H * W} - {0}):
        out, near = oracle.budget_guided_interpolation(X, n)
        h, w = oracle.interpolation_grid(n, H, W)
        for k in range(n):
            i, j = divmod(k, w)
            sy, sx = _pos(i, H, h), _pos(j, W, w)
            assert abs(out[k, 0] - (a * sy + b * sx + c)) < 1e-12
            ny = min(H - 1, int(np.floor((i + 0.5) * H / h)))
            nx = min(W - 1, int(np.floor((j + 0.5) * W / w)))
            assert near[k] == ny * W + nx


@pytest.mark.parametrize("H,W", SHAPES)
def test_matches_torch_interpolate(H, W):
    rng = np.random.default_rng(7 + H + W)
    X = rng.standard_normal((H, W, 4))
    for n in sorted({1, 5, 12, 20, (H * W + 1) // 2, H * W} & set(range(1, H * W + 1))):
        h, w = oracle.interpolation_grid(n, H, W)
        ref = torch.nn.functional.interpolate(torch.from_numpy(X).permute(2, 0, 1)[None], size=(h, w),
                                              mode="bilinear", align_corners=False)[0].permute(1, 2, 0)
        ref = ref.reshape(h * w, 4).numpy()[:n]
        out, _ = oracle.budget_guided_interpolation(X, n)
        np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("H,W", SHAPES)
def test_matches_map_coordinates(H, W):
    rng = np.random.default_rng(11 + H * W)
    X = rng.standard_normal((H, W, 2))
    for n in sorted({1, 3, 10, H * W // 2 + 1} & set(range(1, H * W + 1))):
        h, w = oracle.interpolation_grid(n, H, W)
        ks = np.arange(n)
        ys = np.array([_pos(k // w, H, h) for k in ks])
        xs = np.array([_pos(k % w, W, w) for k in ks])
        ref = np.stack([scipy.ndimage.map_coordinates(X[:, :, c], [ys, xs], order=1, mode="nearest")
                        for c in range(2)], axis=1)
        out, _ = oracle.budget_guided_interpolation(X, n)
        np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-12)


def test_condense_interp_keeps_budgets_and_interpolates_the_modulated_map():
    rng = np.random.default_rng(3)
    T, H, W, C, Q = 4, 5, 6, 16, 3
    X = rng.standard_normal((T, H, W, C))
    q = rng.standard_normal((Q, C))
    sel = oracle.condense(X, q, 40, levels=1, lam=1.5)
    itp = oracle.condense(X, q, 40, levels=1, lam=1.5, assign="interp")
    assert np.array_equal(sel["budget"], itp["budget"]) and np.array_equal(sel["offset"], itp["offset"])
    for t in range(T):
        n = int(itp["budget"][t])
        if n == 0:
            continue
        Xt = oracle.wavelet_spatial_modulator(X[t], itp["M"][t].reshape(H, W), 1.5)
        out, near = oracle.budget_guided_interpolation(Xt, n)
        o0, o1 = itp["offset"][t], itp["offset"][t + 1]
        assert np.array_equal(itp["tokens"][o0:o1], out)
        assert np.array_equal(itp["index"][o0:o1], t * H * W + near)
