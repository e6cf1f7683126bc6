"""Find, per workload, the first seed whose oracle decisions clear the tie margins.

Run from the repository root:  python tests/golden/find_seeds.py [workload ...]
Prints one line per workload; the accepted seeds are recorded in the workload
table of paper_2607_23265_amd/synth.py.  Calls only the input generator and the
oracle.
"""
import os
import sys

sys.path.insert(0, os.path.join(os.path.dirname(__file__), ".."))
sys.path.insert(0, os.path.join(os.path.dirname(__file__), "..", ".."))

import oracle  # noqa: E402
import margins  # noqa: E402
from paper_2607_23265_amd import synth  # noqa: E402


def accepted_seed(wl, start=0, tries=100):
    for seed in range(start, start + tries):
        inp = synth.generate(wl, seed)
        out = oracle.condense(inp.X_f64(), inp.query_f64(), wl.B, wl.levels, wl.lam, wl.tau)
        bad = margins.check(out, wl.N, wl.B, wl.tau)
        print(f"  {wl.name} seed {seed}: {'ok' if not bad else bad[:3]}", flush=True)
        if not bad:
            return seed
    raise RuntimeError(f"no seed within {tries} tries for {wl.name}")


if __name__ == "__main__":
    names = sys.argv[1:] or synth.ORDER
    for name in names:
        print(name, accepted_seed(synth.WORKLOADS[name]), flush=True)
