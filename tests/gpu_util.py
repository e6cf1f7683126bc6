"""Shared helpers of the GPU parity tests."""
import functools

import numpy as np

import margins
import oracle
from paper_2607_23265_amd import synth

# Float tolerances.  Inputs in bf16 with fp32 accumulation: 2e-3; fp32 inputs:
# 1e-5.  A bf16 output adds its own rounding (half an ulp, 2^-8 relative) to
# the fp32 result's error: 2^-8 * (1 + 2e-3) + 2e-3 < 6e-3.
#
# Relative error is floored: err = |got - want| / max(|want|, f * max|want|).
# An output computed in fp32 from operands as large as max|want| carries an
# absolute error of a few fp32 ulps of max|want| (~1e-7 * max|want|), however
# small the output itself; the floor f makes tol * f * max|want| a bound well
# above that: f = 1e-3 for tol 2e-3 (2e-6 * max) and f = 0.1 for tol 1e-5
# (1e-6 * max).
TOL_BF16_IN = 2e-3
TOL_F32_IN = 1e-5
TOL_BF16_OUT = 6e-3
FLOOR = {TOL_BF16_IN: 1e-3, TOL_BF16_OUT: 1e-3, TOL_F32_IN: 0.1}


def rel_err(got, want, floor_frac=1e-3):
    """Max over elements of |got - want| / max(|want|, floor_frac * max|want|) (0 for empty)."""
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    if want.size == 0:
        return 0.0
    floor = floor_frac * float(np.max(np.abs(want)))
    den = np.maximum(np.abs(want), floor if floor > 0 else 1e-30)
    return float(np.max(np.abs(got - want) / den))


def unfloored_err(got, want):
    """Max over the elements with want != 0 of |got - want| / |want| (0 when there are none)."""
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    nz = want != 0
    if not nz.any():
        return 0.0
    return float(np.max(np.abs(got[nz] - want[nz]) / np.abs(want[nz])))


def needed_floor(got, want, tol):
    """Smallest floor fraction f with rel_err(got, want, f) <= tol (0 when no element needs one)."""
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    if want.size == 0:
        return 0.0
    m = float(np.max(np.abs(want)))
    diff = np.abs(got - want)
    over = diff > tol * np.abs(want)
    if not over.any():
        return 0.0
    return float(np.max(diff[over])) / (tol * m) if m > 0 else float("inf")


def within(got, want, tol, label="tensor"):
    """rel_err with the floor that belongs to `tol` is at most `tol`.  Prints the floored and the
    unfloored maximum error and the smallest floor that would still pass, so the run's log records
    how far below the bar each tensor is."""
    floored = rel_err(got, want, FLOOR[tol])
    print(f"[err] {label}: floored {floored:.3e} (floor {FLOOR[tol]:g} x max, bar {tol:g}), "
          f"unfloored {unfloored_err(got, want):.3e}, needed floor {needed_floor(got, want, tol):.2e}", flush=True)
    return floored <= tol


def tol_for(in_dtype):
    return TOL_BF16_IN if in_dtype == "bf16" else TOL_F32_IN


@functools.lru_cache(maxsize=6)
def workload_case(name):
    """Inputs and oracle output of a named workload (cached per test session)."""
    wl = synth.WORKLOADS[name]
    inp = synth.generate(wl)
    out = oracle.condense(inp.X_f64(), inp.query_f64(), wl.B, wl.levels, wl.lam, wl.tau)
    return wl, inp, out


def bf16_round(x):
    """Round float64 values to the bf16 grid (via float32, nearest-even)."""
    return synth.bf16_bits_to_f64(synth.f32_to_bf16_bits(np.asarray(x, dtype=np.float32)))


def check_margins(out, N, B, tau):
    """Margin violations of an oracle run, ignoring exact ties (resolved by index on both sides)."""
    bad = []
    for kind, detail in margins.check(out, N, B, tau):
        if kind == "selection" and detail[2] == 0.0:
            continue
        bad.append((kind, detail))
    return bad
