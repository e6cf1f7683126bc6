"""WaveZip token-condensation pass -- plain CPU oracle in float64 NumPy.

TEST INFRASTRUCTURE ONLY.  This module is the slow, obviously-correct statement
of what the GPU path computes.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import it; the product path never does, and it
shares no code, constants or helpers with the HIP kernels.

Source: "WaveZip: Wavelet-Driven Space-Time Decoupling for Video Token
Condensation", Sec. 3 (Method).  Every function names the passage it follows.
Points where the paper is silent or ambiguous follow these readings:

  * multi-token query: a score against the query is the maximum over query
    tokens of the cosine (Sec. 3.2.1 defines one global query embedding);
  * a cosine with a zero-norm vector is 0;
  * the rank-preserving normalisation of Eq. (7) is a per-frame min-max, and a
    frame whose scores are all equal gets M = 0; gamma of Sec. 3.2.2 is the
    same min-max over all T frames (0 when degenerate);
  * frame 0 is always retained by the frame filter (delta_1 = 0 by Eq. (8));
    delta is clamped to [0, 2] against rounding;
  * the down-sampling of the gate in Eq. (10) is pair averaging, applied once
    per decomposition level; J temporal levels gate every detail level;
  * odd-length signals are extended by repeating the last sample before every
    Haar step (half-point symmetric extension), and cropped after synthesis;
  * db4 and bior4.4 (the paper's spatial default and its basis ablation) use
    the filter-bank conventions stated above `filter_bank`: half-sample
    symmetric extension, floor((L + F - 1) / 2) coefficients a level, outputs
    cropped; the gate is pooled to a subband's length by adaptive average
    pooling (bins floor(i L / n) .. ceil((i + 1) L / n) - 1);
  * the orthonormal Haar filters are used in 1-D and, separably, in 2-D; the
    2-D transform is the single-level Haar version of Eq. (12)-(15); the
    multi-level variant (spatial_levels > 1) gates level j's details by the
    saliency map pooled j times;
  * Eq. (16)'s Round is realised as a capped largest-remainder (Hamilton)
    apportionment so that Eq. (5) (budgets sum to B) holds with 0 <= n <= N;
    remainder ties go to the smaller frame index; if every weight is zero the
    weights are uniform;
  * the budget-guided interpolation of Eq. (17) is replaced by keeping the n_m
    tokens of largest saliency a (ties -> smaller index), emitted in raster
    order; frames are concatenated in temporal order as in Eq. (19);
  * the interpolation itself (assign="interp"), Psi of Eq. (17), whose grid
    the paper does not give: n tokens are the first n cells, in raster order,
    of an h' x w' grid keeping the frame's aspect ratio (h0 = the integer
    nearest sqrt(n H / W), halves up, within [1, H]; w' = min(W, ceil(n / h0));
    h' = ceil(n / w'), so that no grid row is empty); cell (i, j) is the
    bilinear interpolation of the modulated map at the half-pixel centre
    ((2i + 1) H / (2 h') - 1/2, (2j + 1) W / (2 w') - 1/2), negative
    coordinates clamped to 0, the last row / column repeated past the edge;
    its index is the token nearest that point (halves up).

Arrays: X is [T, H, W, C] and query is [Q, C], both float64 holding the exact
values of the (already cast) inputs.  Indices are 0-based.  parity pinned:
every function below is checked by tests against closed forms, invariants,
hand-derived cases and a pure-Python brute force.
"""
import numpy as np

_INV_SQRT2 = 1.0 / np.sqrt(2.0)


# ---------------------------------------------------------------------------
# Cross-Modal Scorer, similarity branch (Sec. 3.2.1)
# ---------------------------------------------------------------------------

def cosine_matrix(U, V):
    """cos(u_i, v_j) for rows of U [n, C] and V [m, C]; 0 where a norm is 0."""
    dots = U @ V.T
    nu = np.sqrt(np.sum(U * U, axis=1))
    nv = np.sqrt(np.sum(V * V, axis=1))
    den = nu[:, None] * nv[None, :]
    out = np.zeros_like(dots)
    nz = den > 0
    out[nz] = dots[nz] / den[nz]
    return out


def token_saliency(X, query):
    """Spatial saliency a_{t,n} (Sec. 3.2.1, token-wise cosine with the query).

    Returns a [T, H*W]: max over query tokens of cos(x_{t,n}, q_j).
    """
    T, H, W, C = X.shape
    cos = cosine_matrix(X.reshape(T * H * W, C), query)
    return cos.max(axis=1).reshape(T, H * W)


def pooled_features(X):
    """Spatially average-pooled frame features v-bar_t (Sec. 3.2.1, Eq. (8))."""
    return X.mean(axis=(1, 2))


def frame_relevance(vbar, query):
    """Temporal relevance r_t: cosine of the pooled frame with the query (Sec. 3.2.1)."""
    return cosine_matrix(vbar, query).max(axis=1)


# ---------------------------------------------------------------------------
# Visual Change Estimator (Sec. 3.2.2)
# ---------------------------------------------------------------------------

def visual_change(vbar):
    """delta_t of Eq. (8): cosine distance of adjacent pooled features; delta_1 = 0."""
    T = vbar.shape[0]
    delta = np.zeros(T)
    for t in range(1, T):
        c = cosine_matrix(vbar[t:t + 1], vbar[t - 1:t])[0, 0]
        delta[t] = min(max(1.0 - c, 0.0), 2.0)
    return delta


def min_max(v):
    """Min-max normalisation to [0, 1]; all-equal input gives zeros."""
    lo, hi = np.min(v), np.max(v)
    if hi > lo:
        return (v - lo) / (hi - lo)
    return np.zeros_like(v)


def temporal_gate(delta):
    """gamma_t = min-max normalised delta over the temporal axis (Sec. 3.2.2)."""
    return min_max(delta)


def retained_frames(delta, tau):
    """Frame Filter of Sec. 3.2.2: keep t with delta_t >= tau, frame 0 always."""
    return [0] + [t for t in range(1, len(delta)) if delta[t] >= tau]


def saliency_map(a_t):
    """M_t of Eq. (7): per-frame rank-preserving (min-max) normalisation of a."""
    return min_max(a_t)


# ---------------------------------------------------------------------------
# Haar wavelet (Eq. (9), (11), (12), (15))
# ---------------------------------------------------------------------------

def _extend_even(x, axis):
    """Repeat the last sample along `axis` when its length is odd."""
    if x.shape[axis] % 2 == 0:
        return x
    last = np.take(x, [x.shape[axis] - 1], axis=axis)
    return np.concatenate([x, last], axis=axis)


def haar_analysis(x, axis=0):
    """One orthonormal Haar analysis step along `axis` -> (approximation, detail).

    A_k = (x_{2k} + x_{2k+1}) / sqrt(2),  D_k = (x_{2k} - x_{2k+1}) / sqrt(2),
    after extending an odd-length axis by its last sample.
    """
    xe = _extend_even(np.asarray(x, dtype=np.float64), axis)
    n = xe.shape[axis]
    even = np.take(xe, np.arange(0, n, 2), axis=axis)
    odd = np.take(xe, np.arange(1, n, 2), axis=axis)
    return (even + odd) * _INV_SQRT2, (even - odd) * _INV_SQRT2


def haar_synthesis(A, D, length, axis=0):
    """Inverse of `haar_analysis`: interleave (A+D)/sqrt(2), (A-D)/sqrt(2), crop to `length`."""
    even = (A + D) * _INV_SQRT2
    odd = (A - D) * _INV_SQRT2
    shape = list(A.shape)
    shape[axis] = 2 * A.shape[axis]
    out = np.empty(shape)
    idx = [slice(None)] * len(shape)
    idx[axis] = slice(0, None, 2)
    out[tuple(idx)] = even
    idx[axis] = slice(1, None, 2)
    out[tuple(idx)] = odd
    idx[axis] = slice(0, length)
    return out[tuple(idx)]


def pair_average(g):
    """Average pooling by pairs (the down-sampling P of Eq. (10)); odd length repeats the last entry."""
    ge = _extend_even(np.asarray(g, dtype=np.float64), 0)
    return 0.5 * (ge[0::2] + ge[1::2])


# ---------------------------------------------------------------------------
# Wavelet Temporal Allocator (Eq. (9)-(11))
# ---------------------------------------------------------------------------

def wavelet_temporal_allocator(R, Gamma, levels):
    """Rectified relevance R-tilde.

    Level j = 1..J: (A_j, D_j) = DWT(A_{j-1}) with A_0 = R (Eq. (9)); the gate is
    pooled to the detail resolution, Gamma-bar_j = P(Gamma-bar_{j-1}), and
    D-tilde_j = Gamma-bar_j * D_j (Eq. (10)); the inverse DWT then rebuilds the
    sequence level by level (Eq. (11)).  With J = 1 this is the paper's
    single-level WTA.
    """
    A = np.asarray(R, dtype=np.float64)
    g = np.asarray(Gamma, dtype=np.float64)
    lengths, details = [], []
    for _ in range(levels):
        lengths.append(A.shape[0])
        A, D = haar_analysis(A)
        g = pair_average(g)
        details.append(g * D)
    for j in reversed(range(levels)):
        A = haar_synthesis(A, details[j], lengths[j])
    return A


# ---------------------------------------------------------------------------
# Token Assigner: frame budgets (Eq. (16) with the constraint of Eq. (5))
# ---------------------------------------------------------------------------

def allocate_budget(r_tilde, B, N):
    """Integer budgets n_m >= 0 for the retained frames, sum = min(B, L*N), each <= N.

    Quota q_m = R * w_m / sum(w) with w = max(r-tilde, 0) (Eq. (16)).  A frame whose
    quota reaches N is fixed at N and the rest of the budget is re-apportioned
    among the others; otherwise every frame gets floor(q_m) and the leftover
    tokens go to the largest fractional parts, smaller index first on ties.
    """
    return allocate_budget_trace(r_tilde, B, N)[0]


def allocate_budget_trace(r_tilde, B, N):
    """`allocate_budget` plus a record of its last apportionment round.

    The record holds the quotas `q` of the frames `active` in that round, the
    number `left` of leftover tokens handed out by fractional part, whether the
    all-zero-weight rule (`uniform`) or the spread-after-capping rule
    (`reactivated`) fired, the frames fixed at N (`capped`), and the quotas of
    every round in order (`rounds`, the capping rounds included).
    """
    L = len(r_tilde)
    n = np.zeros(L, dtype=np.int64)
    trace = dict(q=np.zeros(0), active=np.zeros(0, dtype=np.int64), left=0,
                 uniform=False, reactivated=False, capped=np.zeros(L, dtype=bool), rounds=[])
    if B >= L * N:
        n[:] = N
        trace["capped"][:] = True
        return n, trace
    w = np.maximum(np.asarray(r_tilde, dtype=np.float64), 0.0)
    if np.sum(w) == 0.0:
        w = np.ones(L)
        trace["uniform"] = True
    capped = np.zeros(L, dtype=bool)
    active = w > 0
    R = int(B)
    while R > 0:
        if not np.any(active):
            # every positively weighted frame is full: spread the rest evenly
            active = ~capped
            w = np.where(capped, 0.0, 1.0)
            trace["reactivated"] = True
        idx = np.nonzero(active)[0]
        q = R * w[idx] / np.sum(w[idx])
        trace["rounds"].append(q)
        full = q >= N
        if np.any(full):
            n[idx[full]] = N
            capped[idx[full]] = True
            active[idx[full]] = False
            R -= N * int(np.count_nonzero(full))
            continue
        base = np.floor(q)
        left = R - int(np.sum(base))
        frac = q - base
        order = np.lexsort((idx, -frac))       # frac descending, then index ascending
        n[idx] = base.astype(np.int64)
        n[idx[order[:left]]] += 1
        trace.update(q=q, active=idx, left=left)
        R = 0
    trace["capped"] = capped
    return n, trace


# ---------------------------------------------------------------------------
# Wavelet Spatial Modulator (Eq. (12)-(15)) with the single-level Haar basis
# ---------------------------------------------------------------------------

def haar_analysis_2d(F):
    """Single-level separable 2-D Haar of F [H, W, ...] -> (LL, LH, HL, HH) (Eq. (12)).

    The first letter is the filter along the height axis, the second along the width.
    """
    lo_w, hi_w = haar_analysis(F, axis=1)
    LL, HL = haar_analysis(lo_w, axis=0)
    LH, HH = haar_analysis(hi_w, axis=0)
    return LL, LH, HL, HH


def haar_synthesis_2d(LL, LH, HL, HH, H, W):
    """Inverse of `haar_analysis_2d`, cropped to H x W (Eq. (15))."""
    lo_w = haar_synthesis(LL, HL, H, axis=0)
    hi_w = haar_synthesis(LH, HH, H, axis=0)
    return haar_synthesis(lo_w, hi_w, W, axis=1)


def block_average(Mhw):
    """Average-pool an H x W map to the Haar subband grid (P of Eq. (13))."""
    Me = _extend_even(_extend_even(np.asarray(Mhw, dtype=np.float64), 0), 1)
    return 0.25 * (Me[0::2, 0::2] + Me[0::2, 1::2] + Me[1::2, 0::2] + Me[1::2, 1::2])


def wavelet_spatial_modulator(F, Mhw, lam, levels=1):
    """X-tilde_m for one frame F [H, W, C] with saliency map Mhw [H, W].

    G_m = lam * P(M_m) (Eq. (13)); the three detail subbands are multiplied by G_m
    (Eq. (14)) and the frame is rebuilt by the inverse transform (Eq. (15)); the
    approximation LL is left unchanged.  With levels = J > 1 (the multi-level
    variant of the ablation space) the approximation is decomposed again J - 1
    times; level j's details are gated by lam times M pooled j times (odd sizes
    repeat the last row / column at every level) and the levels are rebuilt from
    the coarsest.
    """
    H, W = Mhw.shape
    LL = np.asarray(F, dtype=np.float64)
    M = np.asarray(Mhw, dtype=np.float64)
    shapes, gated = [], []
    for _ in range(levels):
        shapes.append(LL.shape[:2])
        LL, LH, HL, HH = haar_analysis_2d(LL)
        M = block_average(M)
        G = (lam * M)[:, :, None]
        gated.append((G * LH, G * HL, G * HH))
    for (h, w), (LH, HL, HH) in zip(reversed(shapes), reversed(gated)):
        LL = haar_synthesis_2d(LL, LH, HL, HH, h, w)
    return LL


# ---------------------------------------------------------------------------
# Wavelet bases beyond Haar: db4 (the paper's spatial default, Sec. 3.2.3 and
# Sec. 4.1) and bior4.4 (the basis ablation of Sec. 4.3)
# ---------------------------------------------------------------------------
# A filter bank is (dec_lo, dec_hi, rec_lo, rec_hi), all of one even length F.
# One analysis step of a signal x of length L gives n = floor((L + F - 1) / 2)
# coefficients per band,
#     a[k] = sum_j dec_lo[j] x~[2k + 1 - j],   d[k] = sum_j dec_hi[j] x~[2k + 1 - j],
# x~ the half-sample symmetric extension of x (x~[-1-i] = x[i],
# x~[L+i] = x[L-1-i], repeated with period 2L).  Synthesis rebuilds
#     x[i] = sum_k rec_lo[i + F - 2 - 2k] a[k] + rec_hi[i + F - 2 - 2k] d[k]
# (terms with the filter index outside [0, F) dropped) for i < 2n - F + 2,
# which is L or L + 1 and is cropped to L.  For Haar this is the step above
# (d[k] = (x[2k] - x[2k+1]) / sqrt 2, an odd length repeating its last sample).
# The high-pass filters follow from the low-pass ones:
#     rec_hi[k] = (-1)^k dec_lo[k],   dec_hi[k] = -(-1)^k rec_lo[k].

def daubechies_lowpass(N):
    """Daubechies' minimum-phase low-pass filter with N vanishing moments (2N taps, sum sqrt 2).

    Its squared frequency response is cos^2N(w/2) P(sin^2(w/2)) with
    P(y) = sum_{k<N} C(N-1+k, k) y^k; each root y of P gives the pair of zeros
    z, 1/z of z^2 - (2 - 4y) z + 1, and the one inside the unit circle is kept.
    Taps in the order h_0, h_1, ... of the published tables.
    """
    from math import comb
    roots_y = np.roots([comb(N - 1 + k, k) for k in range(N)][::-1])
    poly = np.array([1.0 + 0j])
    for _ in range(N):
        poly = np.convolve(poly, [1.0, 1.0])
    for y in roots_y:
        pair = np.roots([1.0, -(2.0 - 4.0 * y), 1.0])
        poly = np.convolve(poly, [1.0, -pair[np.argmin(np.abs(pair))]])
    h = np.real(poly)
    return h * np.sqrt(2.0) / h.sum()


def cdf_lowpasses():
    """The Cohen-Daubechies-Feauveau 9/7 pair behind bior4.4: (analysis 9 taps, synthesis 7 taps).

    The same polynomial P(y) with N = 4 splits between the two filters: the
    complex pair of roots (four zeros) goes with (1 + z)^4 into the analysis
    low-pass, the real root (two zeros) with (1 + z)^4 into the synthesis
    low-pass; both symmetric, each normalised to sum sqrt 2.
    """
    from math import comb
    roots_y = np.roots([comb(3 + k, k) for k in range(4)][::-1])
    ana, syn = np.array([1.0 + 0j]), np.array([1.0 + 0j])
    for _ in range(4):
        ana, syn = np.convolve(ana, [1.0, 1.0]), np.convolve(syn, [1.0, 1.0])
    for y in roots_y:
        quad = [1.0, -(2.0 - 4.0 * y), 1.0]
        if abs(y.imag) > 1e-12:
            ana = np.convolve(ana, quad)
        else:
            syn = np.convolve(syn, quad)
    ana, syn = np.real(ana), np.real(syn)
    return ana * np.sqrt(2.0) / ana.sum(), syn * np.sqrt(2.0) / syn.sum()


def filter_bank(basis):
    """(dec_lo, dec_hi, rec_lo, rec_hi) of "haar", "db4" or "bior4.4" (conventions above)."""
    if basis == "haar":
        rec_lo = np.array([1.0, 1.0]) * _INV_SQRT2
        dec_lo = rec_lo[::-1].copy()
    elif basis == "db4":
        rec_lo = daubechies_lowpass(4)
        dec_lo = rec_lo[::-1].copy()
    elif basis == "bior4.4":
        ana, syn = cdf_lowpasses()
        dec_lo, rec_lo = np.zeros(10), np.zeros(10)
        dec_lo[1:10] = ana
        rec_lo[1:8] = syn
    else:
        raise ValueError(f"unknown wavelet basis {basis!r}")
    sign = (-1.0) ** np.arange(len(dec_lo))
    return dec_lo, -sign * rec_lo, rec_lo, sign * dec_lo


def _symmetric_index(i, L):
    """Index into x of position i of its half-sample symmetric extension."""
    i = np.mod(i, 2 * L)
    return np.where(i < L, i, 2 * L - 1 - i)


def dwt_step(x, bank, axis=0, mode="symmetric"):
    """One analysis step along `axis` -> (approximation, detail) (Eq. (9), Eq. (12) per axis).

    mode "symmetric": the extension above (floor((L + F - 1) / 2) coefficients);
    mode "periodization": x~ periodic with period L (L even, L / 2 coefficients),
    the orthogonal form used only to check energy preservation.
    """
    dec_lo, dec_hi = bank[0], bank[1]
    x = np.asarray(x, dtype=np.float64)
    L, F = x.shape[axis], len(dec_lo)
    n = (L + F - 1) // 2 if mode == "symmetric" else L // 2
    a = np.zeros(x.shape[:axis] + (n,) + x.shape[axis + 1:])
    d = np.zeros_like(a)
    for j in range(F):
        pos = 2 * np.arange(n) + 1 - j
        idx = _symmetric_index(pos, L) if mode == "symmetric" else np.mod(pos, L)
        xs = np.take(x, idx, axis=axis)
        a += dec_lo[j] * xs
        d += dec_hi[j] * xs
    return a, d


def idwt_step(a, d, bank, length, axis=0):
    """Synthesis step inverting `dwt_step` (mode symmetric), cropped to `length` (Eq. (11), Eq. (15))."""
    rec_lo, rec_hi = bank[2], bank[3]
    a = np.asarray(a, dtype=np.float64)
    d = np.asarray(d, dtype=np.float64)
    n, F = a.shape[axis], len(rec_lo)
    m = 2 * n - F + 2
    out = np.zeros(a.shape[:axis] + (m,) + a.shape[axis + 1:])
    idx = [slice(None)] * out.ndim
    for i in range(m):
        acc = np.zeros(np.take(a, [0], axis=axis).shape)
        for k in range(n):
            f = i + F - 2 - 2 * k
            if 0 <= f < F:
                acc = acc + rec_lo[f] * np.take(a, [k], axis=axis) + rec_hi[f] * np.take(d, [k], axis=axis)
        idx[axis] = slice(i, i + 1)
        out[tuple(idx)] = acc
    idx[axis] = slice(0, length)
    return out[tuple(idx)]


def adaptive_average(v, n, axis=0):
    """Average pooling of `axis` (length L) to n outputs: output i is the mean of
    positions floor(i L / n) .. ceil((i + 1) L / n) - 1 (the down-sampling of
    Eq. (10) and Eq. (13) to a subband's resolution)."""
    v = np.asarray(v, dtype=np.float64)
    L = v.shape[axis]
    parts = []
    for i in range(n):
        lo, hi = (i * L) // n, -((-(i + 1) * L) // n)
        parts.append(np.take(v, np.arange(lo, hi), axis=axis).mean(axis=axis, keepdims=True))
    return np.concatenate(parts, axis=axis)


def wavelet_temporal_allocator_bank(R, Gamma, levels, basis):
    """Eq. (9)-(11) with the filter bank of `basis` (the Haar case is `wavelet_temporal_allocator`).

    Level j = 1..J: (A_j, D_j) = dwt_step(A_{j-1}); the gate is pooled to the
    detail length by `adaptive_average` of the previous level's gate (Gamma at
    level 0); D~_j = Gamma-bar_j * D_j; synthesis from the coarsest level, each
    level cropped to the length it had.
    """
    bank = filter_bank(basis)
    A = np.asarray(R, dtype=np.float64)
    g = np.asarray(Gamma, dtype=np.float64)
    lengths, details = [], []
    for _ in range(levels):
        lengths.append(A.shape[0])
        A, D = dwt_step(A, bank)
        g = adaptive_average(g, D.shape[0])
        details.append(g * D)
    for j in reversed(range(levels)):
        A = idwt_step(A, details[j], bank, lengths[j])
    return A


def dwt2_step(F, bank):
    """Single-level separable 2-D analysis of F [H, W, ...] -> (LL, LH, HL, HH) (Eq. (12)),
    the first letter the filter along the height, the second along the width."""
    lo_w, hi_w = dwt_step(F, bank, axis=1)
    LL, HL = dwt_step(lo_w, bank, axis=0)
    LH, HH = dwt_step(hi_w, bank, axis=0)
    return LL, LH, HL, HH


def idwt2_step(LL, LH, HL, HH, bank, H, W):
    """Inverse of `dwt2_step`, cropped to H x W (Eq. (15))."""
    lo_w = idwt_step(LL, HL, bank, H, axis=0)
    hi_w = idwt_step(LH, HH, bank, H, axis=0)
    return idwt_step(lo_w, hi_w, bank, W, axis=1)


def wavelet_spatial_modulator_bank(F, Mhw, lam, basis):
    """X-tilde of Eq. (12)-(15) with the filter bank of `basis`, one level.

    G = lam * P(M), P the adaptive average pooling of the H x W saliency map to
    the subband grid (n_h x n_w); LH, HL and HH are multiplied by G, LL kept,
    and the frame rebuilt and cropped to H x W.
    """
    bank = filter_bank(basis)
    H, W = Mhw.shape
    LL, LH, HL, HH = dwt2_step(F, bank)
    G = lam * adaptive_average(adaptive_average(Mhw, LL.shape[0], axis=0), LL.shape[1], axis=1)
    G = G[:, :, None]
    return idwt2_step(LL, G * LH, G * HL, G * HH, bank, H, W)


# ---------------------------------------------------------------------------
# Token Assigner: selection and concatenation (Eq. (17) replaced, Eq. (19))
# ---------------------------------------------------------------------------

def interpolation_grid(n, H, W):
    """(h', w') of the grid that Psi of Eq. (17) samples for n tokens (reading above).

    h0 is the integer nearest sqrt(n H / W) with halves rounded up, i.e. the largest
    h >= 1 with (2h - 1)^2 W <= 4 n H, capped at H; w' = min(W, ceil(n / h0)) and
    h' = ceil(n / w').
    """
    h0 = 1
    while h0 < H and (2 * (h0 + 1) - 1) ** 2 * W <= 4 * n * H:
        h0 += 1
    w = min(W, -(-n // h0))
    return -(-n // w), w


def _sample(i, L, l):
    """Cell i of l cells over L input samples: the half-pixel centre
    s = (2i + 1) L / (2l) - 1/2 as exact integers (num / den), clamped at 0.
    Returns (i0, i1, weight of i1, nearest sample)."""
    num, den = (2 * i + 1) * L - l, 2 * l
    if num < 0:
        i0, frac = 0, 0.0
    else:
        i0, frac = num // den, (num % den) / den
    return i0, min(i0 + 1, L - 1), frac, min(L - 1, ((2 * i + 1) * L) // (2 * l))


def budget_guided_interpolation(Xt, n):
    """Psi(X-tilde_m, n_m) of Eq. (17) for one modulated frame Xt [H, W, C] (reading above).

    Returns (tokens [n, C], index [n]) with index = h * W + w of the nearest token.
    """
    H, W, C = Xt.shape
    h, w = interpolation_grid(n, H, W)
    out = np.zeros((n, C))
    near = np.zeros(n, dtype=np.int64)
    for k in range(n):
        i, j = divmod(k, w)
        y0, y1, fy, ny = _sample(i, H, h)
        x0, x1, fx, nx = _sample(j, W, w)
        top = (1.0 - fx) * Xt[y0, x0] + fx * Xt[y0, x1]
        bottom = (1.0 - fx) * Xt[y1, x0] + fx * Xt[y1, x1]
        out[k] = (1.0 - fy) * top + fy * bottom
        near[k] = ny * W + nx
    return out, near


def select_tokens(a_t, n_t):
    """Indices of the n_t largest saliency scores (ties -> smaller index), ascending."""
    order = np.lexsort((np.arange(len(a_t)), -np.asarray(a_t)))
    return np.sort(order[:n_t])


def condense(X, query, B, levels=1, lam=1.5, tau=0.0, assign="select", spatial_levels=1,
             temporal_basis="haar", spatial_basis="haar"):
    """The whole pass C(X, Q) of Eq. (4)/(6); returns every intermediate.

    assign: "select" keeps each frame's n_t most salient modulated tokens,
    "interp" interpolates the modulated frame to n_t tokens (Psi of Eq. (17)).
    spatial_levels: levels of the spatial Haar modulator (1 as in Eq. (12)-(15)).
    temporal_basis / spatial_basis: "haar" (the transforms above), "db4" or
    "bior4.4" (the filter banks above; one spatial level, selection only).
    Keys: a [T,N], vbar [T,C], r [T], delta [T], gamma [T], retained (list),
    r_tilde [L], budget [T] (0 for dropped frames), offset [T+1], M [T,N],
    tokens [offset[T], C], index [offset[T]] (flat t*N + h*W + w).
    """
    X = np.asarray(X, dtype=np.float64)
    query = np.asarray(query, dtype=np.float64)
    T, H, W, C = X.shape
    N = H * W
    a = token_saliency(X, query)
    vbar = pooled_features(X)
    r = frame_relevance(vbar, query)
    delta = visual_change(vbar)
    gamma = temporal_gate(delta)
    kept_frames = retained_frames(delta, tau)
    if temporal_basis == "haar":
        r_tilde = wavelet_temporal_allocator(r[kept_frames], gamma[kept_frames], levels)
    else:
        r_tilde = wavelet_temporal_allocator_bank(r[kept_frames], gamma[kept_frames], levels, temporal_basis)
    n_kept = allocate_budget(r_tilde, B, N)
    budget = np.zeros(T, dtype=np.int64)
    budget[kept_frames] = n_kept
    offset = np.concatenate([[0], np.cumsum(budget)]).astype(np.int64)
    M = np.stack([saliency_map(a[t]) for t in range(T)])
    tokens = np.zeros((int(offset[T]), C))
    index = np.zeros(int(offset[T]), dtype=np.int64)
    for t in range(T):
        if budget[t] == 0:
            continue
        if spatial_basis == "haar":
            Xt = wavelet_spatial_modulator(X[t], M[t].reshape(H, W), lam, spatial_levels)
        else:
            Xt = wavelet_spatial_modulator_bank(X[t], M[t].reshape(H, W), lam, spatial_basis)
        if assign == "interp":
            tok_t, near = budget_guided_interpolation(Xt, int(budget[t]))
            tokens[offset[t]:offset[t + 1]] = tok_t
            index[offset[t]:offset[t + 1]] = t * N + near
        else:
            sel = select_tokens(a[t], int(budget[t]))
            tokens[offset[t]:offset[t + 1]] = Xt.reshape(N, C)[sel]
            index[offset[t]:offset[t + 1]] = t * N + sel
    return dict(a=a, vbar=vbar, r=r, delta=delta, gamma=gamma, retained=kept_frames,
                r_tilde=r_tilde, budget=budget, offset=offset, M=M,
                tokens=tokens, index=index)
