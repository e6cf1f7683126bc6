"""The seeded input generator: determinism, the bf16 cast, and the statistics it promises."""
import numpy as np
import torch

from paper_2607_23265_amd import synth


def test_deterministic_per_seed():
    wl = synth.small("t32_14x14_c3584", T=4, C=64, Q=3)
    a, b, c = synth.generate(wl, 5), synth.generate(wl, 5), synth.generate(wl, 6)
    assert np.array_equal(a.X, b.X) and np.array_equal(a.query, b.query)
    assert not np.array_equal(a.X, c.X)


def test_bf16_cast_matches_torch_rne():
    rng = np.random.default_rng(3)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 10,
                        np.array([1.00390625, 1.01171875, -1.00390625, 0.0, -0.0, 3.0e-39], np.float32)])
    ours = synth.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    back = synth.bf16_bits_to_f64(ours)
    assert np.array_equal(back, torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy())


def test_ar1_correlation_and_cuts():
    wl = synth.small("t64_14x14_c3584", T=64, C=256, Q=2, scale_sigma=0.0, dtype="f32")
    inp = synth.generate(wl)
    X = inp.X.astype(np.float64)
    cuts = set(inp.cut_frames)
    lag = [np.corrcoef(X[t].ravel(), X[t - 1].ravel())[0, 1] for t in range(1, wl.T) if t not in cuts]
    assert abs(np.mean(lag) - wl.rho) < 0.01
    at_cut = [np.corrcoef(X[t].ravel(), X[t - 1].ravel())[0, 1] for t in cuts]
    assert all(abs(c) < 0.05 for c in at_cut)
    # stationary variance 1 / (1 - rho^2)
    assert abs(X.var() * (1 - wl.rho ** 2) - 1.0) < 0.05


def test_cut_rate_and_outliers():
    wl = synth.small("t256_27x27_c1152", T=256, H=4, W=4, C=32, Q=2)
    counts = [len(synth.generate(wl, s).cut_frames) for s in range(20)]
    assert abs(np.mean(counts) - 255 / 12) < 3.0
    inp = synth.generate(wl, 0)
    X = synth.bf16_bits_to_f64(inp.X)
    # heavy-tailed outliers: some |x| far beyond what the Gaussian part reaches
    assert np.max(np.abs(X)) > 20.0 / np.sqrt(1 - wl.rho ** 2)


def test_workload_table():
    w = synth.WORKLOADS
    assert [w[n].B for n in synth.ORDER] == [128, 627, 1254, 2163, 9331]
    assert w["t64_14x14_c3584"].levels == 2 and w["t64_14x14_c3584"].x_bytes == 64 * 196 * 3584 * 2
    assert all(w[n].lam == 1.5 and w[n].tau == 0.0 for n in synth.ORDER)
