"""Benchmark of the WaveZip condensation pass (wz_condense) on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--out-dtype bf16|f32]

One step = one wz_condense call over one seeded synthetic input set of the
workload (default: T=64 frames of 14x14 tokens, C=3584 bf16, 32 query tokens,
B=1254, 2 temporal levels).  Inputs are resident in HBM before timing; the
call cycles through enough separate copies of the input (>= 512 MB in all)
that the 256 MB Infinity Cache cannot serve a repeated frame tensor.

The K timed steps run as R back-to-back groups (default 5) with a HIP event
between groups and no synchronisation inside; `ms_per_step` is the median
group's time per step, `ms_per_step_groups` lists every group.

Prints one JSON line: frames condensed per second (value), tokens/s, the
algorithmic HBM rate of the whole call, the roofline of the dominant kernel
(the relevance pass, timed with HIP events on its stream, with the HBM bytes
and MFMA busy share that rocprofv3 counters recorded for the same sources),
the rate of a plain read of the frame tensor on the same device
(`read_ceiling`, the achievable streaming rate beside the 8 TB/s peak), the
CPU oracle's rate on the host (all cores and one thread) as a reported
baseline, (`interp`) the rate with the
budget-guided interpolation forming the tokens instead of selection,
(`bases`) the rates with db4 or bior4.4 spatial modulators and a bior4.4
temporal allocator, (`spatial_levels_2`) the rate with the two-level spatial modulator, and
(`batched`) the rate of wz_condense_batch on several videos of the same
workload per call, and (`queries`) the rate of wz_condense_queries with
several queries over each video per call -- separate modes, not the
headline value.
"""
import argparse
import hashlib
import json
import math
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, HERE)

METRIC = "frames condensed/s and achieved HBM GB/s (T=64, 14×14, C=3584 bf16)"
HBM_PEAK_GBPS = 8000.0
MALL_BYTES = 256 << 20


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="t64_14x14_c3584")
    ap.add_argument("--out-dtype", default="bf16", choices=["bf16", "f32"])
    ap.add_argument("--repeats", type=int, default=5,
                    help="timed groups the K steps are split into (median reported)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="approximate CPU time spent timing the oracle (0 disables)")
    ap.add_argument("--videos", type=int, default=4,
                    help="also time wz_condense_batch on this many videos of the workload per call (0 disables)")
    ap.add_argument("--queries", type=int, default=2,
                    help="also time wz_condense_queries with this many queries per video per call (0 disables)")
    ap.add_argument("--read-calib", type=int, default=0,
                    help="only run this many plain reads of the frame tensor (the read ceiling) and exit")
    ap.add_argument("--copy-calib", type=int, default=0,
                    help="only run this many plain device copies of a frame tensor (the known-size kernel that "
                         "scales HBM byte counters) and exit")
    return ap.parse_args()


def algorithmic_bytes(wl, out_bytes):
    """Bytes the pass must move per call: frames read once, query, condensed rows, indices, budgets."""
    s_in = 2 if wl.dtype == "bf16" else 4
    return (wl.T * wl.N * wl.C * s_in + wl.Q * wl.C * s_in + wl.B * wl.C * out_bytes + 4 * wl.B + 4 * wl.T)


def kernel_sources_sha256():
    """Digest of the kernel and C-ABI sources, to tell whether recorded counters still describe them."""
    h = hashlib.sha256()
    csrc = os.path.join("paper_2607_23265_amd", "csrc")
    files = sorted([os.path.join(csrc, f) for f in os.listdir(os.path.join(HERE, csrc)) if f.endswith((".hip", ".h"))] +
                   [os.path.join("include", f) for f in os.listdir(os.path.join(HERE, "include")) if f.endswith(".h")])
    for f in files:
        h.update(f.encode())
        with open(os.path.join(HERE, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def recorded_counters(workload):
    """rocprofv3 counter figures of the relevance pass for the workload (profiles/), or None when there is
    no record or the kernel sources changed since it was taken: HBM bytes per launch (FETCH_SIZE and
    WRITE_SIZE, scaled by a plain device copy) and the MFMA busy share (SQ_VALU_MFMA_BUSY_CYCLES over
    GRBM_GUI_ACTIVE times the SIMD count)."""
    path = os.path.join(HERE, "profiles", f"relevance_pass_counters_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        rec = json.load(fh)
    if rec.get("kernel_sources_sha256") != kernel_sources_sha256():
        return None
    return rec


def relevance_bytes(wl):
    """Bytes the relevance pass must move: frames and query read once, per-token scores written (the
    per-unit partial sums it also writes are left out, so the rate is a lower bound)."""
    s_in = 2 if wl.dtype == "bf16" else 4
    return wl.T * wl.N * wl.C * s_in + wl.Q * wl.C * s_in + 4 * wl.T * wl.N


def _time_oracle(oracle, X, q, wl, seconds):
    """Whole oracle passes over the same input until ~`seconds` elapse; returns seconds per pass."""
    calls, t0 = 0, time.perf_counter()
    while True:
        oracle.condense(X, q, wl.B, wl.levels, wl.lam, wl.tau)
        calls += 1
        el = time.perf_counter() - t0
        if el >= seconds:
            return el / calls, calls


def cpu_baseline(inp, wl, seconds):
    """Time the CPU oracle (as written) on whole passes over the same input: three timed runs on all the
    host's BLAS threads (median reported) and one run on a single thread, ~`seconds` of CPU time in all."""
    import numpy as np  # noqa: F401
    import oracle
    from threadpoolctl import threadpool_info, threadpool_limits
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    X, q = inp.X_f64(), inp.query_f64()
    runs = [_time_oracle(oracle, X, q, wl, seconds / 4) for _ in range(3)]
    per_pass = sorted(r[0] for r in runs)[1]
    with threadpool_limits(limits=1):
        one, one_calls = _time_oracle(oracle, X, q, wl, seconds / 4)
    return {"value": wl.T / per_pass, "unit": "frames/s", "cores": int(threads), "kind": "oracle",
            "single_thread": {"value": wl.T / one, "unit": "frames/s", "cores": 1, "passes": one_calls},
            "sample": f"median of 3 timed runs of whole passes of the float64 NumPy oracle over the same {wl.name} "
                      f"input ({wl.T} frames each; {sum(r[1] for r in runs)} passes, "
                      f"{sum(r[0] * r[1] for r in runs):.1f} s) on {threads} BLAS threads, and "
                      f"{one_calls} passes on one thread"}


def timed_groups(stream, fn, steps, groups):
    """Run fn(i) for i < steps as `groups` back-to-back groups on `stream`, a HIP event between groups and
    no synchronisation inside; returns (median ms per call over the groups, per-group ms per call)."""
    import torch
    groups = max(1, min(groups, steps))
    sizes = [steps // groups + (1 if g < steps % groups else 0) for g in range(groups)]
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(groups + 1)]
    ev[0].record(stream)
    i = 0
    for g, n in enumerate(sizes):
        for _ in range(n):
            fn(i)
            i += 1
        ev[g + 1].record(stream)
    torch.cuda.synchronize()
    per = [ev[g].elapsed_time(ev[g + 1]) / sizes[g] for g in range(groups)]
    return sorted(per)[(groups - 1) // 2], per


def read_ceiling(Xs, stream, steps):
    """Plain streaming read of the frame tensor (the library's wz_probe_stream_read), cycling through the
    input copies; returns (us per read, GB/s)."""
    import torch
    from paper_2607_23265_amd import wavezip as wz
    n = len(Xs)
    sink = torch.empty(4096, dtype=torch.int32, device=Xs[0].device)
    for i in range(8):
        wz.probe_stream_read(Xs[i % n], sink)
    ms, _ = timed_groups(stream, lambda i: wz.probe_stream_read(Xs[i % n], sink), steps, 5)
    nbytes = Xs[0].numel() * Xs[0].element_size()
    return ms * 1e3, nbytes / (ms * 1e-3) / 1e9


def stream_of(dev):
    import torch
    return torch.cuda.current_stream(dev)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for {args.gpus}); the pass is single-GPU by design.",
              file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2607_23265_amd import synth
    from paper_2607_23265_amd import wavezip as wz

    wl = synth.WORKLOADS[args.workload]
    out_dtype = wz.WZ_BF16 if args.out_dtype == "bf16" else wz.WZ_F32
    p = wz.problem_of(wl, out_dtype)
    dev = "cuda:0"
    torch.cuda.set_device(0)
    inp = synth.generate(wl)
    X0, q0 = wz.to_device(inp, dev)
    nsets = max(1, math.ceil(2 * MALL_BYTES / X0.numel() / X0.element_size()))
    Xs = [X0] + [X0.clone() for _ in range(nsets - 1)]
    qs = [q0] + [q0.clone() for _ in range(nsets - 1)]
    if args.read_calib:
        us, gbps = read_ceiling(Xs, stream_of(dev), args.read_calib)
        print(json.dumps({"calibration": "plain read", "bytes_read": X0.numel() * X0.element_size(),
                          "us_per_read": us, "gbps": gbps, "reads": args.read_calib}), flush=True)
        return
    if args.copy_calib:
        dst = [torch.empty_like(X0) for _ in range(2)]
        for i in range(args.copy_calib):
            dst[i % 2].copy_(Xs[i % nsets])
        torch.cuda.synchronize()
        print(json.dumps({"calibration": "device copy", "bytes_read": X0.numel() * X0.element_size(),
                          "bytes_written": X0.numel() * X0.element_size(), "copies": args.copy_calib}), flush=True)
        return
    ws = wz.new_workspace(p, dev)
    out = wz._out_tokens(p, dev)
    stream = torch.cuda.current_stream(dev)

    def step(i):
        wz.condense(p, Xs[i % nsets], qs[i % nsets], ws=ws, out=out)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ms_step, ms_groups = timed_groups(stream, step, args.steps, args.repeats)
    wall = time.perf_counter() - t0

    # dominant kernel: the relevance pass over X (k_relevance_tok), launched alone through
    # wz_relevance_pass, back to back on the same stream
    a = torch.empty(wl.T * wl.N, dtype=torch.float32, device=dev)
    import ctypes
    L = wz.lib()
    cfg = p.config()
    sp = ctypes.c_void_p(stream.cuda_stream)

    def rel(i):
        st = L.wz_relevance_pass(ctypes.byref(cfg), wz._ptr(Xs[i % nsets]), wz._ptr(qs[i % nsets]), wz._ptr(a),
                                 wz._ptr(ws), ws.numel(), sp)
        if st != 0:
            raise wz.WZError(st, "wz_relevance_pass")

    for i in range(args.warmup):
        rel(i)
    torch.cuda.synchronize()
    k1_ms, k1_groups = timed_groups(stream, rel, args.steps, args.repeats)
    k1_bytes = relevance_bytes(wl)
    k1_gbps = k1_bytes / (k1_ms * 1e-3) / 1e9
    rc_us, rc_gbps = read_ceiling(Xs, stream, args.steps)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    batched = None
    if args.videos > 1:
        # several videos per call (wz_condense_batch): distinct copies of the input so that no video's
        # frames are served from the Infinity Cache of another call
        V = args.videos
        vsets = max(2, math.ceil(2 * MALL_BYTES / (V * X0.numel() * X0.element_size())))
        XB = [torch.stack([Xs[(i * V + v) % nsets] for v in range(V)]) for i in range(vsets)]
        QB = [torch.stack([qs[(i * V + v) % nsets] for v in range(V)]) for i in range(vsets)]
        wsb = torch.empty(V * ws.numel(), dtype=torch.uint8, device=dev)
        dt = torch.float32 if out_dtype == wz.WZ_F32 else torch.bfloat16
        outb = (torch.empty((V, p.B, p.C), dtype=dt, device=dev), torch.empty((V, p.B), dtype=torch.int32, device=dev))
        for i in range(args.warmup):
            wz.condense_batch(p, XB[i % vsets], QB[i % vsets], ws=wsb, out=outb)
        torch.cuda.synchronize()
        bsteps = max(1, args.steps // V)
        ev0.record(stream)
        for i in range(bsteps):
            wz.condense_batch(p, XB[i % vsets], QB[i % vsets], ws=wsb, out=outb)
        ev1.record(stream)
        torch.cuda.synchronize()
        b_ms = ev0.elapsed_time(ev1) / bsteps
        batched = {"videos": V, "calls": bsteps, "ms_per_call": b_ms,
                   "frames_per_s": V * wl.T / (b_ms * 1e-3),
                   "hbm_gbps": V * algorithmic_bytes(wl, 2 if out_dtype == wz.WZ_BF16 else 4) / (b_ms * 1e-3) / 1e9}
        del XB, QB, wsb, outb

    queries = None
    if args.queries > 1:
        # several queries over each video per call (wz_condense_queries): query g is the
        # workload's query with its channels rotated by 8 g
        G = args.queries
        QG = [torch.stack([qs[i % nsets].roll(8 * g, dims=-1) for g in range(G)]).contiguous()
              for i in range(nsets)]
        wsq = torch.empty(G * ws.numel(), dtype=torch.uint8, device=dev)
        dt = torch.float32 if out_dtype == wz.WZ_F32 else torch.bfloat16
        outq = (torch.empty((G, p.B, p.C), dtype=dt, device=dev), torch.empty((G, p.B), dtype=torch.int32, device=dev))
        for i in range(args.warmup):
            wz.condense_queries(p, Xs[i % nsets], QG[i % nsets], ws=wsq, out=outq)
        torch.cuda.synchronize()
        ev0.record(stream)
        for i in range(args.steps):
            wz.condense_queries(p, Xs[i % nsets], QG[i % nsets], ws=wsq, out=outq)
        ev1.record(stream)
        torch.cuda.synchronize()
        q_ms = ev0.elapsed_time(ev1) / args.steps
        queries = {"queries": G, "calls": args.steps, "ms_per_call": q_ms,
                   "queries_per_pass_over_x": min(G, 64 // wl.Q) if wl.dtype == "bf16" and wl.Q <= 64 else 1,
                   "query_frames_per_s": G * wl.T / (q_ms * 1e-3),
                   "vs_separate_calls": G * ms_step / q_ms}
        del QG, wsq, outq

    # the same pass with the budget-guided interpolation forming the tokens (cfg.assign = WZ_INTERP)
    pi = wz.problem_of(wl, out_dtype, assign=wz.WZ_INTERP)
    for i in range(args.warmup):
        wz.condense(pi, Xs[i % nsets], qs[i % nsets], ws=ws, out=out)
    torch.cuda.synchronize()
    ev0.record(stream)
    for i in range(args.steps):
        wz.condense(pi, Xs[i % nsets], qs[i % nsets], ws=ws, out=out)
    ev1.record(stream)
    torch.cuda.synchronize()
    i_ms = ev0.elapsed_time(ev1) / args.steps
    interp = {"ms_per_step": i_ms, "frames_per_s": wl.T / (i_ms * 1e-3)}
    # and with the longer wavelet bases: db4 / bior4.4 spatial modulators, a bior4.4 temporal allocator
    def mode_rate(pm):
        wsm = wz.new_workspace(pm, dev)
        for i in range(args.warmup):
            wz.condense(pm, Xs[i % nsets], qs[i % nsets], ws=wsm, out=out)
        torch.cuda.synchronize()
        m_ms, _ = timed_groups(stream, lambda i: wz.condense(pm, Xs[i % nsets], qs[i % nsets], ws=wsm, out=out),
                               args.steps, args.repeats)
        return {"ms_per_step": m_ms, "frames_per_s": wl.T / (m_ms * 1e-3)}

    bases = {"spatial_db4": mode_rate(wz.problem_of(wl, out_dtype, spatial_basis=wz.WZ_DB4)),
             "spatial_bior4.4": mode_rate(wz.problem_of(wl, out_dtype, spatial_basis=wz.WZ_BIOR44)),
             "temporal_bior4.4": mode_rate(wz.problem_of(wl, out_dtype, temporal_basis=wz.WZ_BIOR44))}
    # and with the two-level spatial modulator (cfg.spatial_levels = 2)
    p2 = wz.problem_of(wl, out_dtype, spatial_levels=2)
    ws2 = wz.new_workspace(p2, dev)
    for i in range(args.warmup):
        wz.condense(p2, Xs[i % nsets], qs[i % nsets], ws=ws2, out=out)
    torch.cuda.synchronize()
    ev0.record(stream)
    for i in range(args.steps):
        wz.condense(p2, Xs[i % nsets], qs[i % nsets], ws=ws2, out=out)
    ev1.record(stream)
    torch.cuda.synchronize()
    l_ms = ev0.elapsed_time(ev1) / args.steps
    levels2 = {"ms_per_step": l_ms, "frames_per_s": wl.T / (l_ms * 1e-3)}

    out_bytes = 2 if out_dtype == wz.WZ_BF16 else 4
    call_bytes = algorithmic_bytes(wl, out_bytes)
    counters = recorded_counters(wl.name)
    frames_s = wl.T / (ms_step * 1e-3)
    line = {
        "metric": METRIC,
        "value": frames_s,
        "unit": "frames/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "T": wl.T, "H": wl.H, "W": wl.W, "C": wl.C, "Q": wl.Q, "B": wl.B,
                   "levels": wl.levels, "lambda": wl.lam, "tau": wl.tau, "in_dtype": wl.dtype,
                   "out_dtype": args.out_dtype, "seed": wl.seed, "input_copies": nsets},
        "tokens_per_s": wl.T * wl.N / (ms_step * 1e-3),
        "hbm_gbps": call_bytes / (ms_step * 1e-3) / 1e9,
        "hbm_frac": call_bytes / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBPS,
        "bytes_per_step": call_bytes,
        "wall_s": wall,
        "ms_per_step_groups": ms_groups,
        "roofline": {"kernel": "k_relevance_tok (wz_relevance_pass: the one pass over the frames)",
                     "bound": "hbm", "achieved": k1_gbps,
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": k1_gbps / HBM_PEAK_GBPS,
                     "traffic": counters["traffic_bytes_per_launch"] if counters else None,
                     "mfma_busy": counters["mfma_busy_frac"] if counters else None,
                     "bytes_per_launch": k1_bytes, "us_per_launch": k1_ms * 1e3,
                     "us_per_launch_groups": [m * 1e3 for m in k1_groups]},
        "read_ceiling": {"what": "wz_probe_stream_read: a plain streaming read of the frame tensor",
                         "us": rc_us, "gbps": rc_gbps, "frac_of_peak": rc_gbps / HBM_PEAK_GBPS},
    }
    line["interp"] = interp
    line["bases"] = bases
    line["spatial_levels_2"] = levels2
    if batched:
        line["batched"] = batched
    if queries:
        line["queries"] = queries
    if args.cpu_seconds > 0:
        line["cpu_baseline"] = cpu_baseline(inp, wl, args.cpu_seconds)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
