"""Tie margins for the pass's discrete decisions (test infrastructure).

The GPU computes scores in float32 and the oracle in float64, so integer
outputs (budgets, kept-token indices) can only be compared bit-exactly on
inputs whose decisions are not within rounding of a tie.  `check` lists every
decision of the oracle's run that falls inside its margin; an input is usable
for exact parity when the list is empty.

Decisions and margins (oracle float64 values):
  selection boundary, per frame   a_(n) - a_(n+1)        >= M_A
  saliency / gate ranges          max - min               >= M_A or exactly 0
  remainder cut-off               frac_(left) - frac_(left+1) >= M_Q tokens
  cap (every round)               |q_t - N|               >= M_Q tokens
  all-weights-zero switch         |max r_tilde|           >= M_R
  weight signs (re-activation)    |r_tilde_m|             >= M_R
  frame filter (tau > 0)          |delta_t - tau|         >= M_D
"""
import numpy as np

import oracle

M_A = 1e-6
M_Q = 1e-3
M_R = 1e-6
M_D = 1e-6


def check(out, N, B, tau=0.0):
    """Return a list of (decision, detail) pairs that violate a margin.

    `out` is the dict returned by `oracle.condense`; N tokens per frame; B the budget.
    """
    bad = []
    a = out["a"]
    T = a.shape[0]
    for t in range(T):
        n = int(out["budget"][t])
        s = np.sort(a[t])[::-1]
        if 0 < n < N and s[n - 1] - s[n] < M_A:
            bad.append(("selection", (t, n, float(s[n - 1] - s[n]))))
        rng = s[0] - s[-1]
        if 0 < rng < M_A:
            bad.append(("saliency_range", (t, float(rng))))
    d = out["delta"]
    drange = float(np.max(d) - np.min(d))
    if 0 < drange < M_D:
        bad.append(("delta_range", drange))
    if tau > 0:
        close = np.abs(d[1:] - tau) < M_D
        if np.any(close):
            bad.append(("frame_filter", np.nonzero(close)[0] + 1))
    rt = out["r_tilde"]
    L = len(rt)
    if L and abs(float(np.max(rt))) < M_R:
        bad.append(("zero_weight_switch", float(np.max(rt))))
    _, trace = oracle.allocate_budget_trace(rt, int(B), N)
    if trace["reactivated"] and np.any(np.abs(rt) < M_R):
        bad.append(("weight_sign", float(np.min(np.abs(rt)))))
    for k, qr in enumerate(trace["rounds"]):
        near = np.abs(qr - N) < M_Q
        if np.any(near):
            bad.append(("cap", (k, float(np.min(np.abs(qr - N))))))
    q, left = trace["q"], trace["left"]
    if 0 < left < len(q):
        frac = np.sort(q - np.floor(q))[::-1]
        if frac[left - 1] - frac[left] < M_Q:
            bad.append(("remainder", (left, float(frac[left - 1] - frac[left]))))
    return bad
