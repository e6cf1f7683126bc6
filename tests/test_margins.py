"""The workloads' recorded seeds give inputs whose discrete decisions clear the tie margins."""
import pytest

import margins
import oracle
from paper_2607_23265_amd import synth


@pytest.mark.parametrize("name", synth.ORDER)
def test_recorded_seed_clears_margins(name):
    wl = synth.WORKLOADS[name]
    inp = synth.generate(wl)
    out = oracle.condense(inp.X_f64(), inp.query_f64(), wl.B, wl.levels, wl.lam, wl.tau)
    assert int(out["budget"].sum()) == wl.B
    assert margins.check(out, wl.N, wl.B, wl.tau) == []
