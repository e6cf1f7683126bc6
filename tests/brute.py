"""Pure-Python restatement of the WaveZip pass for tiny inputs (test infrastructure).

Written independently of the NumPy oracle, in scalar loops and with different
formulations where one exists, so that a slip in either shows up as a
disagreement:

* 2-D Haar: the explicit 2x2 butterflies LL = (p00+p01+p10+p11)/2, ... instead
  of the separable transform;
* temporal Haar: explicit per-level lists with the last sample repeated;
* budget: quotas in exact rational arithmetic (fractions.Fraction) and an
  explicit "largest remainders" sort of (fraction, index) tuples;
* selection: a sort of (-a, n) tuples.

Inputs are nested lists: X[t][h][w][c], query[j][c].  Same readings of the
paper as the oracle (max over query tokens, cos = 0 for a zero vector, min-max
normalisations, frame 0 always retained, last-sample extension, capped
largest-remainder apportionment, top-n selection in raster order).
"""
import math
from fractions import Fraction


def _dot(u, v):
    s = 0.0
    for a, b in zip(u, v):
        s += a * b
    return s


def _cos(u, v):
    nu = math.sqrt(_dot(u, u))
    nv = math.sqrt(_dot(v, v))
    if nu == 0.0 or nv == 0.0:
        return 0.0
    return _dot(u, v) / (nu * nv)


def _minmax(vals):
    lo, hi = min(vals), max(vals)
    if hi > lo:
        return [(v - lo) / (hi - lo) for v in vals]
    return [0.0 for _ in vals]


def _haar_levels(seq, gate, levels):
    s = math.sqrt(2.0)
    approx = list(seq)
    g = list(gate)
    stack = []
    for _ in range(levels):
        n = len(approx)
        if n % 2:
            approx = approx + [approx[-1]]
            g = g + [g[-1]]
        A = [(approx[2 * k] + approx[2 * k + 1]) / s for k in range(len(approx) // 2)]
        D = [(approx[2 * k] - approx[2 * k + 1]) / s for k in range(len(approx) // 2)]
        g = [(g[2 * k] + g[2 * k + 1]) / 2 for k in range(len(g) // 2)]
        stack.append((n, [gk * dk for gk, dk in zip(g, D)]))
        approx = A
    for n, Dt in reversed(stack):
        rebuilt = []
        for a, d in zip(approx, Dt):
            rebuilt.append((a + d) / s)
            rebuilt.append((a - d) / s)
        approx = rebuilt[:n]
    return approx


def _apportion(weights, B, N):
    L = len(weights)
    if B >= L * N:
        return [N] * L
    w = [Fraction(max(x, 0.0)) for x in weights]
    if sum(w) == 0:
        w = [Fraction(1)] * L
    n = [0] * L
    fixed = [False] * L
    R = B
    while R > 0:
        live = [m for m in range(L) if not fixed[m] and w[m] > 0]
        if not live:
            live = [m for m in range(L) if not fixed[m]]
            w = [Fraction(0) if fixed[m] else Fraction(1) for m in range(L)]
        total = sum(w[m] for m in live)
        quota = {m: R * w[m] / total for m in live}
        over = [m for m in live if quota[m] >= N]
        if over:
            for m in over:
                n[m] = N
                fixed[m] = True
            R -= N * len(over)
            continue
        floors = {m: quota[m].numerator // quota[m].denominator for m in live}
        for m in live:
            n[m] = floors[m]
        left = R - sum(floors.values())
        ranked = sorted(live, key=lambda m: (-(quota[m] - floors[m]), m))
        for m in ranked[:left]:
            n[m] += 1
        R = 0
    return n


def condense(X, query, B, levels=1, lam=1.5, tau=0.0):
    T, H, W = len(X), len(X[0]), len(X[0][0])
    C = len(X[0][0][0])
    N = H * W
    tokens = [[X[t][n // W][n % W] for n in range(N)] for t in range(T)]
    a = [[max(_cos(x, q) for q in query) for x in tokens[t]] for t in range(T)]
    pooled = [[sum(tokens[t][n][c] for n in range(N)) / N for c in range(C)] for t in range(T)]
    r = [max(_cos(pooled[t], q) for q in query) for t in range(T)]
    delta = [0.0] + [min(2.0, max(0.0, 1.0 - _cos(pooled[t], pooled[t - 1]))) for t in range(1, T)]
    gamma = _minmax(delta)
    kept = [t for t in range(T) if t == 0 or delta[t] >= tau]
    r_tilde = _haar_levels([r[t] for t in kept], [gamma[t] for t in kept], levels)
    n_kept = _apportion(r_tilde, B, N)
    budget = [0] * T
    for t, n in zip(kept, n_kept):
        budget[t] = n
    out_tokens, out_index = [], []
    for t in range(T):
        if budget[t] == 0:
            continue
        M = _minmax(a[t])
        ranked = sorted(range(N), key=lambda n: (-a[t][n], n))
        chosen = sorted(ranked[:budget[t]])
        for n in chosen:
            h, w = n // W, n % W
            i0, j0 = h - h % 2, w - w % 2
            rows = [i0, min(i0 + 1, H - 1)]
            cols = [j0, min(j0 + 1, W - 1)]
            gate = lam * sum(M[rr * W + cc] for rr in rows for cc in cols) / 4.0
            row = []
            for c in range(C):
                p00 = X[t][rows[0]][cols[0]][c]
                p01 = X[t][rows[0]][cols[1]][c]
                p10 = X[t][rows[1]][cols[0]][c]
                p11 = X[t][rows[1]][cols[1]][c]
                LL = (p00 + p01 + p10 + p11) / 2
                LH = gate * (p00 - p01 + p10 - p11) / 2
                HL = gate * (p00 + p01 - p10 - p11) / 2
                HH = gate * (p00 - p01 - p10 + p11) / 2
                sh = 1 if h % 2 else 0
                sw = 1 if w % 2 else 0
                sign_w = -1 if sw else 1
                sign_h = -1 if sh else 1
                row.append((LL + sign_w * LH + sign_h * HL + sign_w * sign_h * HH) / 2)
            out_tokens.append(row)
            out_index.append(t * N + n)
    return dict(a=a, r=r, delta=delta, gamma=gamma, retained=kept, r_tilde=r_tilde,
                budget=budget, tokens=out_tokens, index=out_index)


# ---------------------------------------------------------------------------
# One level of a filter-bank DWT, for the db4 / bior4.4 modulators: scalar
# loops over an explicitly built extended list (the oracle indexes an
# extension rule instead), synthesis by scattering each coefficient's
# filter-weighted contribution (the oracle gathers per output sample).
# ---------------------------------------------------------------------------

def dwt_bank(x, dec_lo, dec_hi):
    """(a, d) of list x: a[k] = sum_j dec_lo[j] * e[2k + 1 - j + pad], e the list x
    mirrored (half-sample) by pad = len(filter) - 1 samples at each end."""
    L, F = len(x), len(dec_lo)
    pad = F - 1
    e = []
    for i in range(-pad, L + pad):
        j = i
        while j < 0 or j >= L:  # reflect about the half-sample points -1/2 and L - 1/2
            j = -1 - j if j < 0 else 2 * L - 1 - j
        e.append(x[j])
    n = (L + F - 1) // 2
    a = [sum(dec_lo[j] * e[2 * k + 1 - j + pad] for j in range(F)) for k in range(n)]
    d = [sum(dec_hi[j] * e[2 * k + 1 - j + pad] for j in range(F)) for k in range(n)]
    return a, d


def idwt_bank(a, d, rec_lo, rec_hi, length):
    """Inverse of dwt_bank: coefficient k adds rec_lo[f] * a[k] + rec_hi[f] * d[k] to
    sample 2k + f - (F - 2) for every filter position f; samples outside [0, length) dropped."""
    F = len(rec_lo)
    out = [0.0] * length
    for k in range(len(a)):
        for f in range(F):
            i = 2 * k + f - (F - 2)
            if 0 <= i < length:
                out[i] += rec_lo[f] * a[k] + rec_hi[f] * d[k]
    return out
