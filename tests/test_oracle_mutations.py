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


def _daub_max_phase(N):
    # the zeros outside the unit circle (maximum phase) instead of inside
    h = W._orig["daubechies_lowpass"](N)
    return h[::-1].copy()


def _bank_highpass_sign(basis):
    dec_lo, dec_hi, rec_lo, rec_hi = W._orig["filter_bank"](basis)
    return dec_lo, dec_hi, rec_lo, -rec_hi


def _dwt_zero_extension(x, bank, axis=0, mode="symmetric"):
    # zero padding instead of the symmetric extension
    dec_lo, dec_hi = bank[0], bank[1]
    x = np.asarray(x, dtype=np.float64)
    L, F = x.shape[axis], len(dec_lo)
    n = (L + F - 1) // 2 if mode == "symmetric" else L // 2
    a = np.zeros(x.shape[:axis] + (n,) + x.shape[axis + 1:])
    d = np.zeros_like(a)
    for j in range(F):
        pos = 2 * np.arange(n) + 1 - j
        ok = (pos >= 0) & (pos < L)
        xs = np.take(x, np.clip(pos, 0, L - 1), axis=axis)
        shape = [1] * x.ndim
        shape[axis] = n
        xs = xs * ok.reshape(shape)
        a += dec_lo[j] * xs
        d += dec_hi[j] * xs
    return a, d


def _dwt_even_phase(x, bank, axis=0, mode="symmetric"):
    # coefficients taken at the even positions 2k - j instead of 2k + 1 - j
    dec_lo, dec_hi = bank[0], bank[1]
    x = np.asarray(x, dtype=np.float64)
    L, F = x.shape[axis], len(dec_lo)
    n = (L + F - 1) // 2 if mode == "symmetric" else L // 2
    a = np.zeros(x.shape[:axis] + (n,) + x.shape[axis + 1:])
    d = np.zeros_like(a)
    for j in range(F):
        pos = 2 * np.arange(n) - j
        idx = W._symmetric_index(pos, L) if mode == "symmetric" else np.mod(pos, L)
        xs = np.take(x, idx, axis=axis)
        a += dec_lo[j] * xs
        d += dec_hi[j] * xs
    return a, d


def _adaptive_floor_both(v, n, axis=0):
    v = np.asarray(v, dtype=np.float64)
    L = v.shape[axis]
    parts = [np.take(v, np.arange((i * L) // n, max((i * L) // n + 1, ((i + 1) * L) // n)), axis=axis)
             .mean(axis=axis, keepdims=True) for i in range(n)]
    return np.concatenate(parts, axis=axis)


def _wta_bank_gate_approx(R, Gamma, levels, basis):
    # the gate applied to the approximation instead of the detail
    bank = W.filter_bank(basis)
    A = np.asarray(R, dtype=np.float64)
    g = np.asarray(Gamma, dtype=np.float64)
    lengths, details = [], []
    for _ in range(levels):
        lengths.append(A.shape[0])
        A, D = W.dwt_step(A, bank)
        g = W.adaptive_average(g, D.shape[0])
        A = g * A
        details.append(D)
    for j in reversed(range(levels)):
        A = W.idwt_step(A, details[j], bank, lengths[j])
    return A


def _wsm_bank_gate_ll(F, Mhw, lam, basis):
    bank = W.filter_bank(basis)
    H, Wd = Mhw.shape
    LL, LH, HL, HH = W.dwt2_step(F, bank)
    G = lam * W.adaptive_average(W.adaptive_average(Mhw, LL.shape[0], axis=0), LL.shape[1], axis=1)
    G = G[:, :, None]
    return W.idwt2_step(G * LL, G * LH, G * HL, G * HH, bank, H, Wd)


def _wsm_bank_gate_axes_swapped(F, Mhw, lam, basis):
    bank = W.filter_bank(basis)
    H, Wd = Mhw.shape
    LL, LH, HL, HH = W.dwt2_step(F, bank)
    G = lam * W.adaptive_average(W.adaptive_average(Mhw, LL.shape[1], axis=0), LL.shape[0], axis=1)
    G = G[:, :, None]
    if G.shape[:2] != LL.shape[:2]:
        G = G.transpose(1, 0, 2)
    return W.idwt2_step(LL, G * LH, G * HL, G * HH, bank, H, Wd)


def _idwt2_bands_swapped(LL, LH, HL, HH, bank, H, Wd):
    return W._orig["idwt2_step"](LL, HL, LH, HH, bank, H, Wd)


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
    "daubechies_max_phase": ("daubechies_lowpass", _daub_max_phase),
    "bank_highpass_sign": ("filter_bank", _bank_highpass_sign),
    "dwt_zero_extension": ("dwt_step", _dwt_zero_extension),
    "dwt_even_phase": ("dwt_step", _dwt_even_phase),
    "adaptive_average_floor_ends": ("adaptive_average", _adaptive_floor_both),
    "wta_bank_gate_on_approximation": ("wavelet_temporal_allocator_bank", _wta_bank_gate_approx),
    "wsm_bank_gates_LL": ("wavelet_spatial_modulator_bank", _wsm_bank_gate_ll),
    "wsm_bank_gate_axes_swapped": ("wavelet_spatial_modulator_bank", _wsm_bank_gate_axes_swapped),
    "idwt2_bands_swapped": ("idwt2_step", _idwt2_bands_swapped),
}


@pytest.fixture(autouse=True)
def _originals():
    W._orig = {name: getattr(W, name) for name, _ in
               [(n, None) for n in ("haar_analysis", "haar_synthesis", "allocate_budget_trace", "haar_analysis_2d",
                                    "interpolation_grid", "daubechies_lowpass", "filter_bank", "idwt2_step")]}
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
