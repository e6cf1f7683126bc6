"""Planted mistakes in the CPU oracle must be caught by at least one pin.

Each mutation replaces one oracle function by a copy with a plausible slip (a
dropped term, a wrong sign or index, a swapped operand).  The pins of
pins.py are then run; the test passes when some pin fails an assertion (a pin
that merely crashes on the mutant does not count).  Everything runs on the CPU.
"""
import numpy as np
import pytest

import oracle
import pins
from oracle import wavezip_oracle as W

S2 = 1.0 / np.sqrt(2.0)


def _analysis_detail_sign(x, axis=0):
    A, D = W._orig["haar_analysis"](x, axis)
    return A, -D


def _synthesis_swapped(A, D, length, axis=0):
    return W._orig["haar_synthesis"](A, -D, length, axis)


def _extend_with_zero(x, axis):
    if x.shape[axis] % 2 == 0:
        return x
    z = np.zeros_like(np.take(x, [0], axis=axis))
    return np.concatenate([x, z], axis=axis)


def _pair_first(g):
    ge = W._extend_even(np.asarray(g, dtype=np.float64), 0)
    return ge[0::2].copy()


def _wta_gate_on_approx(R, Gamma, levels):
    A = np.asarray(R, dtype=np.float64)
    g = np.asarray(Gamma, dtype=np.float64)
    lengths, details = [], []
    for _ in range(levels):
        lengths.append(A.shape[0])
        A, D = W.haar_analysis(A)
        g = W.pair_average(g)
        A = g * A
        details.append(D)
    for j in reversed(range(levels)):
        A = W.haar_synthesis(A, details[j], lengths[j])
    return A


def _budget_round(r_tilde, B, N):
    w = np.maximum(np.asarray(r_tilde, dtype=np.float64), 0.0)
    if w.sum() == 0:
        w = np.ones(len(w))
    n = np.minimum(np.round(B * w / w.sum()), N).astype(np.int64)
    return n, dict(q=np.zeros(0), active=np.zeros(0, dtype=np.int64), left=0,
                   uniform=False, reactivated=False, capped=np.zeros(len(w), bool))


def _budget_larger_index_first(r_tilde, B, N):
    rev = np.asarray(r_tilde)[::-1]
    n, tr = W._orig["allocate_budget_trace"](rev, B, N)
    return n[::-1].copy(), tr


def _budget_no_cap(r_tilde, B, N):
    return W._orig["allocate_budget_trace"](r_tilde, B, 10 ** 9)


def _bands_swapped(F):
    LL, LH, HL, HH = W._orig["haar_analysis_2d"](F)
    return LL, HL, LH, HH


def _wsm_gate_all(F, Mhw, lam, levels=1):
    # the approximation band gated too, at every level
    LL = np.asarray(F, dtype=np.float64)
    M = np.asarray(Mhw, dtype=np.float64)
    shapes, gated = [], []
    for _ in range(levels):
        shapes.append(LL.shape[:2])
        LL, LH, HL, HH = W.haar_analysis_2d(LL)
        M = W.block_average(M)
        G = (lam * M)[:, :, None]
        LL = G * LL
        gated.append((G * LH, G * HL, G * HH))
    for (h, w), (LH, HL, HH) in zip(reversed(shapes), reversed(gated)):
        LL = W.haar_synthesis_2d(LL, LH, HL, HH, h, w)
    return LL


def _block_max(Mhw):
    Me = W._extend_even(W._extend_even(np.asarray(Mhw, dtype=np.float64), 0), 1)
    return np.maximum(np.maximum(Me[0::2, 0::2], Me[0::2, 1::2]), np.maximum(Me[1::2, 0::2], Me[1::2, 1::2]))


def _saliency_mean_over_query(X, query):
    T, H, Wd, C = X.shape
    return W.cosine_matrix(X.reshape(T * H * Wd, C), query).mean(axis=1).reshape(T, H * Wd)


def _change_without_one_minus(vbar):
    d = np.zeros(vbar.shape[0])
    for t in range(1, vbar.shape[0]):
        d[t] = W.cosine_matrix(vbar[t:t + 1], vbar[t - 1:t])[0, 0]
    return d


def _cosine_unnormalised_rhs(U, V):
    nu = np.sqrt(np.sum(U * U, axis=1))
    out = (U @ V.T) / np.where(nu > 0, nu, 1.0)[:, None]
    return out


def _select_ascending(a_t, n_t):
    order = np.lexsort((np.arange(len(a_t)), np.asarray(a_t)))
    return np.sort(order[:n_t])


def _minmax_degenerate_ones(v):
    lo, hi = np.min(v), np.max(v)
    return (v - lo) / (hi - lo) if hi > lo else np.ones_like(v)


def _filter_drops_first(delta, tau):
    return [t for t in range(len(delta)) if delta[t] >= tau and (t > 0 or tau <= 0)] or [0]


def _sample_corners(i, L, l):
    # align-corners sampling instead of half-pixel centres
    s = i * (L - 1) / (l - 1) if l > 1 else 0.0
    i0 = int(np.floor(s))
    return i0, min(i0 + 1, L - 1), s - i0, min(L - 1, int(np.floor(s + 0.5)))


def _grid_swap(n, H, Wd):
    # rows and columns of the grid exchanged
    w, h = W._orig["interpolation_grid"](n, Wd, H)
    return min(h, H), min(w, Wd)


def _wsm_level2_unpooled_gate(F, Mhw, lam, levels=1):
    # level 2 gated by the level-1 gate subsampled (every other entry) instead
    # of the saliency map pooled a second time
    LL = np.asarray(F, dtype=np.float64)
    M = W.block_average(Mhw)
    shapes, gated = [], []
    for j in range(levels):
        shapes.append(LL.shape[:2])
        LL, LH, HL, HH = W.haar_analysis_2d(LL)
        if j > 0:
            Me = W._extend_even(W._extend_even(M, 0), 1)
            M = Me[0::2, 0::2]
        G = (lam * M)[:, :, None]
        gated.append((G * LH, G * HL, G * HH))
    for (h, w), (LH, HL, HH) in zip(reversed(shapes), reversed(gated)):
        LL = W.haar_synthesis_2d(LL, LH, HL, HH, h, w)
    return LL


MUTATIONS = {
    "haar_detail_sign": ("haar_analysis", _analysis_detail_sign),
    "haar_synthesis_swapped": ("haar_synthesis", _synthesis_swapped),
    "odd_extension_zero": ("_extend_even", _extend_with_zero),
    "gate_pool_first_sample": ("pair_average", _pair_first),
    "gate_on_approximation": ("wavelet_temporal_allocator", _wta_gate_on_approx),
    "budget_plain_round": ("allocate_budget_trace", _budget_round),
    "budget_tie_larger_index": ("allocate_budget_trace", _budget_larger_index_first),
    "budget_no_cap": ("allocate_budget_trace", _budget_no_cap),
    "bands_swapped": ("haar_analysis_2d", _bands_swapped),
    "wsm_gates_LL": ("wavelet_spatial_modulator", _wsm_gate_all),
    "gate_pool_max": ("block_average", _block_max),
    "saliency_mean_query": ("token_saliency", _saliency_mean_over_query),
    "change_missing_one_minus": ("visual_change", _change_without_one_minus),
    "cosine_missing_norm": ("cosine_matrix", _cosine_unnormalised_rhs),
    "select_smallest": ("select_tokens", _select_ascending),
    "minmax_degenerate_ones": ("min_max", _minmax_degenerate_ones),
    "filter_drops_frame0": ("retained_frames", _filter_drops_first),
    "interp_align_corners": ("_sample", _sample_corners),
    "interp_grid_transposed": ("interpolation_grid", _grid_swap),
    "wsm_level2_unpooled_gate": ("wavelet_spatial_modulator", _wsm_level2_unpooled_gate),
}


@pytest.fixture(autouse=True)
def _originals():
    W._orig = {name: getattr(W, name) for name, _ in
               [(n, None) for n in ("haar_analysis", "haar_synthesis", "allocate_budget_trace", "haar_analysis_2d",
                                    "interpolation_grid")]}
    yield
    del W._orig


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(name, monkeypatch):
    attr, fn = MUTATIONS[name]
    monkeypatch.setattr(W, attr, fn)
    if hasattr(oracle, attr):
        monkeypatch.setattr(oracle, attr, fn)
    caught, crashed = [], []
    for pin in pins.ALL_PINS:
        try:
            pin()
        except AssertionError:
            caught.append(pin.__name__)
        except Exception as e:  # noqa: BLE001 - a crash is not a caught mistake
            crashed.append((pin.__name__, f"{type(e).__name__}: {e}"))
    # only a failed assertion counts: a mutant that merely crashes a pin proves nothing
    assert caught, f"planted mistake {name!r} in {attr} went unnoticed by every pin (crashes: {crashed})"
