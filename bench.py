"""Benchmark of the FastBDT fit/apply hot path on one MI355X.

One step = fbdt_fit of the 500k-event workload (20 features, 256 bins,
depth 3, 100 trees, shrinkage 0.1, sub-sampling 0.5) followed by fbdt_apply
of the fitted forest to the same 500k binned events.  The binned features
are produced once by fbdt_bin before the timed region and stay resident in
HBM.  Prints one JSON line:
  value  = binned event*features per tree layer per second over the step
           (N * d * D * T / step time);
  roofline = the histogram kernel's algorithmic bytes per launch over its
           mean launch duration, from HIP events that the library records
           around every histogram launch on its stream during a second timed
           region of the same steps (events add a few microseconds between
           kernels, so the step time comes from the first region, which
           records none), against 8 TB/s;
  cpu_baseline = the CPU oracle fitting the first trees of the same
           workload on this host, in the same unit.
Also reported, outside the step: "apply" = the 400-tree forest applied to 50M
fresh events (events/s); "fit_workloads" = full fits of the 2M x 40 (200
trees) and 10M x 40 (depth 6, 100 trees) workloads, with the histogram
kernel's mean launch and roofline fraction on each; "section4" = on the
2M x 40 sample, fits with negative event weights and with missing values
against the plain fit, and the per-event and global feature importance.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = ("fit: binned event·features/s per tree layer (HBM GB/s); apply: events/s")
HBM_PEAK_GBS = 8000.0
# integer VALU peak of MI355X: 256 CUs x 4 SIMDs x 16 lanes per clock x 2.4 GHz
VALU_PEAK_GOPS = 256 * 64 * 2.4
APPLY_OPS_PER_NODE_STEP = 4


def measured_traffic():
    """HBM bytes per histogram launch from the committed hardware-counter
    summary, if it was taken on the current kernel source; else None."""
    import hashlib
    src = os.path.join(ROOT, "paper_1609_06119_amd", "csrc", "kernels.hip")
    rec = os.path.join(ROOT, "profiles", "hist_kernel_config2_pmc.json")
    try:
        with open(rec) as fh:
            data = json.load(fh)
        with open(src, "rb") as fh:
            digest = hashlib.sha256(fh.read()).hexdigest()
    except OSError:
        return None
    if data.get("kernels_hip_sha256") != digest:
        return None
    return data.get("bytes_per_launch")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--cpu-trees", type=int, default=100,
                    help="trees of the CPU-oracle baseline sample")
    ap.add_argument("--apply-events", type=int, default=50_000_000,
                    help="fresh events of the apply workload (0 skips it)")
    ap.add_argument("--apply-steps", type=int, default=3,
                    help="timed applies of the 400-tree forest to the fresh events")
    ap.add_argument("--section4", type=int, default=1,
                    help="also time negative weights, missing values and importance (1/0)")
    ap.add_argument("--fit-workloads", default="3,4",
                    help="larger fit workloads also timed and reported (comma list, '' for none)")
    ap.add_argument("--oracle-baseline", type=int, default=1,
                    help="time the CPU oracle per phase on bounded samples of every workload (1/0)")
    ap.add_argument("--phases", type=int, default=1,
                    help="histogram phase timeline and reference passes (1/0)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="after the run, copy a buffer of this size on the device three "
                         "times (reference kernel for hardware byte counters)")
    return ap.parse_args()


def measure_fit_workload(cfg, fb, torch):
    """One full fit of a larger workload (all trees), timed twice: once as
    launched in production (graph replay, no events) for the fit time, once
    with HIP events around every histogram launch for the kernel's roofline."""
    from synth import CONFIGS, make_training_set
    spec = CONFIGS[cfg]
    t0 = time.time()
    ds = make_training_set(cfg)
    d, n = ds["x"].shape
    x = torch.from_numpy(ds["x"]).cuda()
    y = torch.from_numpy(ds["y"]).cuda()
    _, codes = fb.bin(x, spec.n_bins)
    del x, ds
    B, D, T = spec.n_bins, spec.depth, spec.n_trees

    def fit():
        return fb.fit(codes, y, B, D, T, spec.shrinkage, spec.subsample, spec.fit_seed)

    fit()   # warm-up (records the graph)
    torch.cuda.synchronize()
    ts = time.perf_counter()
    model = fit()
    torch.cuda.synchronize()
    fit_s = time.perf_counter() - ts
    # the fitted forest applied to the training events (the general
    # traversal for depth > 3, the two-events-per-lane one below)
    prob = torch.empty(n, dtype=torch.float32, device="cuda")
    fb.apply(model, codes, prob=prob)
    torch.cuda.synchronize()
    ta = time.perf_counter()
    fb.apply(model, codes, prob=prob)
    torch.cuda.synchronize()
    apply_s = time.perf_counter() - ta
    del prob, model
    fb.timing_enable(("histogram", "best_cuts", "route"))
    fit()
    torch.cuda.synchronize()
    hl, hms, hb = fb.timing_read("histogram")
    cl, cms, _ = fb.timing_read("best_cuts")
    rl, rms, _ = fb.timing_read("route")
    fb.timing_enable(())
    del codes, y
    torch.cuda.empty_cache()
    achieved = hb / (hms / 1e3) / 1e9
    return {"workload": f"fit {n} x {d}, {B} bins, depth {D}, {T} trees ({spec.name})",
            "fit_ms": fit_s * 1e3,
            "value": n * d * D * T / fit_s,
            "unit": "event*features/s per tree layer",
            "hist_mean_launch_us": hms * 1e3 / hl,
            "hist_algorithmic_bytes_per_launch": hb / hl,
            "hist_achieved_gbs": achieved,
            "hist_frac": achieved / HBM_PEAK_GBS,
            "cut_scan_mean_launch_us": cms * 1e3 / max(cl, 1),
            "apply_ms": apply_s * 1e3,
            "apply_events_per_s": n / apply_s,
            # layers with more than 4 parents: routing as a pass of its own
            "route_launches": rl,
            "route_mean_launch_us": rms * 1e3 / rl if rl else None,
            "setup_s": round(time.time() - t0, 1)}


def measure_hist_phases(fb, torch, codes, y, spec):
    """Where a histogram launch of the bench workload spends its time.

    One fit with the library's phase timeline on: every workgroup of every
    histogram launch stamps the device's constant-rate clock at entry, once
    the parents' cuts are in LDS, after its first step of events is added,
    after every add and after its partial rows are written.  Per layer, the
    stamps relative to the launch's first entry are averaged over the
    workgroups and then over the trees; "last_*" is the latest workgroup.
    Beside it, the reference passes on the same launch shape (empty
    workgroups; workgroups that only read what the pass reads), timed with
    HIP events like the histogram launches, with the histogram launches of
    the same layer timed the same way."""
    import numpy as np
    B, D, T = spec.n_bins, spec.depth, spec.n_trees
    fb.set_option("hist_timeline", 1)
    try:
        fb.fit(codes, y, B, D, T, spec.shrinkage, spec.subsample, spec.fit_seed)
        torch.cuda.synchronize()
        st, blocks, rate_khz = fb.hist_timeline()
    finally:
        fb.set_option("hist_timeline", 0)
    us = 1e3 / rate_khz
    # stamp columns: entry, cuts in LDS, first step added, adds done, rows
    # written, last wavefront's entry, LDS cleared (wavefront 0)
    cols = {"entry": 0, "last_wave_entry": 5, "lds_cleared": 6, "table": 1, "first_step": 2,
            "adds_done": 3, "rows_written": 4}
    layers = {}
    for layer in range(D):
        acc = {k: [] for k in list(cols) + ["last_entry", "last_rows_written"]}
        for t in range(T):
            rows = st[t * D + layer, :blocks[t * D + layer]].astype(np.int64)
            rows = rows[rows[:, 0] != 0]
            t0 = rows[:, 0].min()
            rel = (rows - t0) * us
            for k, i in cols.items():
                col = rel[:, i][rows[:, i] != 0]
                acc[k].append(col.mean())
            acc["last_entry"].append(rel[:, 0].max())
            acc["last_rows_written"].append(rel[:, 4].max())
        layers[f"layer{layer}"] = {k + "_us": float(np.mean(v)) for k, v in acc.items()}
        layers[f"layer{layer}"]["workgroups"] = int(blocks[layer])
    # reference passes on the launch shapes of layer 0 (no node ids) and of
    # the last layer (node ids read), against the histogram launches
    n = codes.n
    npad = (n + 7) // 8 * 8
    w = torch.zeros(npad, dtype=torch.float32, device="cuda")
    node = torch.zeros(npad, dtype=torch.uint8, device="cuda")
    refs = {}
    for layer in (0, D - 1):
        out = {}
        for kind, name in ((0, "empty"), (1, "read"), (2, "read_up_front")):
            for _ in range(3):
                fb.reference_pass(kind, codes, B, layer, w, node if layer >= 1 else None)
            torch.cuda.synchronize()
            fb.timing_enable(("reference",))
            for _ in range(50):
                fb.reference_pass(kind, codes, B, layer, w, node if layer >= 1 else None)
            torch.cuda.synchronize()
            k, ms, by = fb.timing_read("reference")
            fb.timing_enable(())
            out[f"{name}_mean_launch_us"] = ms * 1e3 / k
            if kind >= 1:
                out[f"{name}_bytes_per_launch"] = by / k
                out[f"{name}_gbs"] = by / (ms / 1e3) / 1e9
        refs[f"layer{layer}"] = out
    fb.timing_enable(("histogram",))
    fb.fit(codes, y, B, D, T, spec.shrinkage, spec.subsample, spec.fit_seed)
    torch.cuda.synchronize()
    hl, hms, _ = fb.timing_read("histogram")
    fb.timing_enable(())
    return {"clock_khz": rate_khz, "phases": layers, "reference": refs,
            "hist_mean_launch_us_same_timing": hms * 1e3 / hl,
            "note": "phase stamps in microseconds after the launch's first workgroup entry"}


def host_info():
    """CPU model, core counts and numpy version of this host."""
    import platform
    import numpy as np
    model = platform.processor() or "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    usable = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    return {"cpu_model": model, "nproc": os.cpu_count(), "usable_cores": usable,
            "numpy": np.__version__, "threads_used": 1}


def _stats(xs):
    import numpy as np
    return {"min": float(np.min(xs)), "mean": float(np.mean(xs)), "max": float(np.max(xs)),
            "repeats": len(xs)}


def measure_oracle_baseline(apply_model=None):
    """The CPU oracle (single-threaded numpy, as it stands) timed per phase
    on bounded samples of every workload: binning of a few features of the
    full sample, a few trees of the fit (per layer: histogram, cumulative
    sums + gains + best cut, routing), and apply; repeated up to 5 times
    (min/mean/max).  The samples are stated with each workload."""
    import numpy as np
    from oracle import fbdt_oracle as O
    from synth import CONFIGS, make_apply_chunk, make_training_set
    # workload -> (events used, features binned, trees fitted, repeats)
    plan = {1: (None, None, None, 5), 2: (None, 2, 5, 5), 3: (None, 2, 1, 5),
            4: (1_000_000, 2, 1, 1)}
    out = {}
    for cfg, (n_ev, nbf, trees, reps) in plan.items():
        spec = CONFIGS[cfg]
        t0 = time.time()
        ds = make_training_set(cfg, n_events=n_ev)
        d, n = ds["x"].shape
        B, D = spec.n_bins, spec.depth
        T = spec.n_trees if trees is None else trees
        jb = d if nbf is None else nbf
        bin_s, fit_s, app_s, steps = [], [], [], []
        for _ in range(reps):
            tb = time.perf_counter()
            O.bin_features(ds["x"][:jb], B)
            bin_s.append((time.perf_counter() - tb) * d / jb)
        _, xb = O.bin_features(ds["x"], B) if jb == d else (None, None)
        if xb is None:
            xb = np.stack([O.encode(ds["x"][j], O.quantile_boundaries(ds["x"][j], B))
                           for j in range(d)])
        del ds["x"]
        for _ in range(reps):
            tm = {}
            tf = time.perf_counter()
            m = O.fit(xb, ds["y"], ds["v"], D, T, spec.shrinkage, spec.subsample,
                      spec.fit_seed, B, timings=tm)
            fit_s.append((time.perf_counter() - tf) / T)
            steps.append(tm)
            ta = time.perf_counter()
            O.apply(m, xb)
            app_s.append((time.perf_counter() - ta) / T)
        layer_us = {}
        for key in steps[0]:
            layer_us[key + "_us_per_tree"] = float(np.mean([st[key] for st in steps])) / T * 1e6
        per_tree = _stats(fit_s)
        out[f"workload{cfg}"] = {
            "sample": ((f"all {n} events" if n == spec.n_events else
                        f"{n} events drawn from the {spec.n_events}-event workload's "
                        f"distribution (same seed)") +
                       f" x {d} features; binning timed on {jb} feature(s) and scaled to {d}; "
                       f"fit of the first {T} of {spec.n_trees} trees; apply of those trees to "
                       f"the {n} events"),
            "bin_s_all_features": _stats(bin_s),
            "fit_s_per_tree": per_tree,
            "fit_s_all_trees_est": per_tree["mean"] * spec.n_trees * spec.n_events / n,
            "value": n * d * D / per_tree["mean"],
            "unit": "event*features/s per tree layer",
            "steps": layer_us,
            "apply_s_per_tree": _stats(app_s),
            "apply_events_per_s_all_trees": n / (np.mean(app_s) * spec.n_trees),
            "setup_s": round(time.time() - t0, 1)}
        print(f"# oracle baseline workload {cfg}: {per_tree['mean']:.3f} s per tree",
              file=sys.stderr, flush=True)
    if apply_model is not None:
        s5 = CONFIGS[5]
        m = 200_000
        xf = make_apply_chunk(0, m)["x"]
        xb = np.stack([O.encode(xf[j], apply_model["boundaries"][j]) for j in range(xf.shape[0])])
        om = O.Model(apply_model["depth"], apply_model["n_bins"], apply_model["n_features"],
                     apply_model["f0"], apply_model["cut_feature"], apply_model["cut_bin"],
                     apply_model["gain"], apply_model["leaf"])
        app = []
        for _ in range(3):
            ta = time.perf_counter()
            O.apply(om, xb)
            app.append(time.perf_counter() - ta)
        out["workload5"] = {
            "sample": f"apply of the fitted {s5.n_trees}-tree forest to {m} of the "
                      f"{s5.apply_events} fresh events (binned by the oracle)",
            "apply_s": _stats(app), "events_per_s": m / float(np.mean(app)),
            "unit": "events/s"}
    return {"host": host_info(), "kind": "oracle", "workloads": out}


def measure_section4(fb, torch):
    """The features of sections 4.1-4.3 on workload 3's sample (2M x 40, 256
    bins, 200 trees of depth 3), each against the plain fit of the same
    sample: a fit with negative event weights (v uniform in [-0.6, 2.5]), a
    fit with missing values (NaN in the float features, features in turn
    0%, 3%, 20% and 60% missing, 255 bins so that code 255 marks them), and
    the per-event and global importance of the plain model.  Times are one
    fit (or call) after a warm-up, host clock around a synchronised call."""
    import numpy as np
    from synth import CONFIGS, make_training_set
    spec = CONFIGS[3]
    t0 = time.time()
    ds = make_training_set(3)
    d, n = ds["x"].shape
    y = torch.from_numpy(ds["y"]).cuda()

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        ts = time.perf_counter()
        out = fn()
        torch.cuda.synchronize()
        return out, (time.perf_counter() - ts) * 1e3

    def fit(codes, n_bins, w=None):
        return lambda: fb.fit(codes, y, n_bins, spec.depth, spec.n_trees, spec.shrinkage,
                              spec.subsample, spec.fit_seed, w=w)

    _, codes = fb.bin(torch.from_numpy(ds["x"]).cuda(), spec.n_bins)
    plain, plain_ms = timed(fit(codes, spec.n_bins))
    v = np.random.default_rng(9).uniform(-0.6, 2.5, n).astype(np.float32)
    _, signed_ms = timed(fit(codes, spec.n_bins, torch.from_numpy(v).cuda()))
    xm = ds["x"].copy()
    rng = np.random.default_rng(7)
    for j in range(d):
        xm[j, rng.random(n) < (0.0, 0.03, 0.2, 0.6)[j % 4]] = np.nan
    _, mcodes = fb.bin(torch.from_numpy(xm).cuda(), 255)
    del xm
    mmodel, missing_ms = timed(fit(mcodes, 255))
    has_inner = "inner" in mmodel.export()
    ei = torch.empty((d, n), dtype=torch.float64, device="cuda")
    _, ei_ms = timed(lambda: fb.event_importance(plain, codes, out=ei))
    _, fi_ms = timed(lambda: fb.feature_importance(plain))
    del ei, codes, mcodes, y
    torch.cuda.empty_cache()
    return {"workload": f"fit {n} x {d}, depth {spec.depth}, {spec.n_trees} trees "
                        f"({spec.name})",
            "plain_fit_ms": plain_ms,
            "negative_weights_fit_ms": signed_ms,
            "missing_values_fit_ms": missing_ms,
            "missing_values_model_has_inner_weights": has_inner,
            "event_importance_ms": ei_ms,
            "event_importance_events_per_s": n / (ei_ms / 1e3),
            "feature_importance_ms": fi_ms,
            "setup_s": round(time.time() - t0, 1)}


def measure_apply_workload(args, apply_x, fb, torch):
    """Workload 5: a 400-tree depth-3 forest fitted on workload 3's 2M x 40
    sample (256 bins), applied to the fresh events (binned with the training
    boundaries, chunk by chunk, into one code buffer).  Returns events/s of
    fbdt_apply from HIP events around each timed launch."""
    from synth import CONFIGS, make_training_set
    s3, s5 = CONFIGS[3], CONFIGS[5]
    t0 = time.time()
    ds = make_training_set(3)
    x3 = torch.from_numpy(ds["x"]).cuda()
    y3 = torch.from_numpy(ds["y"]).cuda()
    bounds, codes3 = fb.bin(x3, s5.n_bins)
    del x3
    model = fb.fit(codes3, y3, s5.n_bins, s5.depth, s5.n_trees, s5.shrinkage, s5.subsample,
                   s5.fit_seed)
    torch.cuda.synchronize()
    fit_s = time.time() - t0
    n = sum(x.shape[1] for _, x in apply_x)
    d = apply_x[0][1].shape[0]
    codes = fb.Codes.empty(d, n)
    for off, x in apply_x:
        m = x.shape[1]
        part = fb.bin_transform(torch.from_numpy(x).cuda(), bounds)
        codes.data[:, off:off + m].copy_(part.data[:, :m])
    del part
    prob = torch.empty(n, dtype=torch.float32, device="cuda")
    fb.apply(model, codes, prob=prob)   # warm-up
    torch.cuda.synchronize()
    fb.timing_enable(("apply",))
    for _ in range(max(1, args.apply_steps)):
        fb.apply(model, codes, prob=prob)
    torch.cuda.synchronize()
    launches, ms, _ = fb.timing_read("apply")
    fb.timing_enable(())
    mean_ms = ms / max(launches, 1)
    del codes
    prob_binned = prob.clone()
    # the same events as float32 values, tested against value thresholds
    # (the training boundaries attached to the model)
    xf = torch.empty((d, n), dtype=torch.float32, device="cuda")
    for off, x in apply_x:
        xf[:, off:off + x.shape[1]].copy_(torch.from_numpy(x))
    model.set_boundaries(bounds)
    fb.apply_float(model, xf, prob=prob)   # warm-up
    torch.cuda.synchronize()
    fb.timing_enable(("apply",))
    for _ in range(max(1, args.apply_steps)):
        fb.apply_float(model, xf, prob=prob)
    torch.cuda.synchronize()
    fl, fms, _ = fb.timing_read("apply")
    fb.timing_enable(())
    same = bool(torch.equal(prob, prob_binned))
    del xf, prob_binned
    f_ms = fms / max(fl, 1)
    gm = model.export()
    oracle_model = {k: gm[k] for k in ("depth", "n_bins", "n_features", "f0", "cut_feature",
                                       "cut_bin", "gain", "leaf")}
    oracle_model["boundaries"] = bounds
    float_out = {"events_per_s": n / (f_ms / 1e3), "launches": fl, "mean_launch_us": f_ms * 1e3,
                 "bytes_per_event": 4 * d + 4,
                 "hbm_gbs": n * (4 * d + 4) / (f_ms / 1e3) / 1e9,
                 "workload": f"the same forest and events as float32 values [{d}][{n}], "
                             "value thresholds (fbdt_apply_float)",
                 "prob_equal_to_binned_apply": same}
    # ALU roofline: the traversal's algorithmic integer work is 4 lane
    # operations per node step (fetch the node's code, compare with the cut,
    # form the child index, select), T * D node steps per event; the peak is
    # MI355X's integer VALU issue rate, 256 CUs x 64 lanes per clock x 2.4 GHz
    ops = n * s5.n_trees * s5.depth * APPLY_OPS_PER_NODE_STEP
    achieved = ops / (mean_ms / 1e3) / 1e9
    return {"events_per_s": n / (mean_ms / 1e3), "launches": launches,
            "mean_launch_us": mean_ms * 1e3,
            "bytes_per_event": d + 4,
            "hbm_gbs": n * (d + 4) / (mean_ms / 1e3) / 1e9,
            "hbm_frac": n * (d + 4) / (mean_ms / 1e3) / 1e9 / HBM_PEAK_GBS,
            "roofline": {"bound": "alu", "kernel": "apply_shallow_kernel<3> (binned)",
                         "achieved": achieved, "peak": VALU_PEAK_GOPS,
                         "unit": "G int32 lane-ops/s", "frac": achieved / VALU_PEAK_GOPS,
                         "ops_per_node_step": APPLY_OPS_PER_NODE_STEP,
                         "node_steps_per_event": s5.n_trees * s5.depth},
            "workload": f"{s5.n_trees}-tree depth-{s5.depth} forest fitted on workload 3 "
                        f"({s3.n_events} x {s3.n_features}, {s5.n_bins} bins) applied to {n} "
                        f"fresh events x {d} uint8 codes; prob float32 out",
            "setup_s": round(fit_s, 1), "float": float_out, "_oracle_model": oracle_model}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported "
              "(the library has no multi-GPU path)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    from synth import CONFIGS, apply_chunks, digest, make_training_set

    # The apply workload's fresh events are drawn first, in worker processes,
    # before this process touches the GPU.
    apply_x = []
    if args.apply_events > 0:
        t0 = time.time()
        apply_x = list(apply_chunks(args.apply_events, workers=16))
        print(f"# apply workload: {args.apply_events} fresh events drawn in "
              f"{time.time() - t0:.1f}s", file=sys.stderr, flush=True)

    import torch

    import paper_1609_06119_amd as fb

    spec = CONFIGS[2]
    t0 = time.time()
    ds = make_training_set(2)
    n, d = ds["x"].shape[1], ds["x"].shape[0]
    B, D, T = spec.n_bins, spec.depth, spec.n_trees
    print(f"# workload: {spec.name}; generated in {time.time() - t0:.1f}s", file=sys.stderr,
          flush=True)

    x = torch.from_numpy(ds["x"]).cuda()
    y = torch.from_numpy(ds["y"]).cuda()
    torch.cuda.synchronize()
    tb = time.perf_counter()
    bounds, codes = fb.bin(x, B)
    torch.cuda.synchronize()
    bin_ms = (time.perf_counter() - tb) * 1e3
    # a second call into the same code buffer (scratch and sort set-up warm)
    tb = time.perf_counter()
    fb.bin(x, B, codes=codes)
    torch.cuda.synchronize()
    bin_warm_ms = (time.perf_counter() - tb) * 1e3
    del x
    prob = torch.empty(n, dtype=torch.float32, device="cuda")

    def step():
        model = fb.fit(codes, y, B, D, T, spec.shrinkage, spec.subsample, spec.fit_seed)
        fb.apply(model, codes, prob=prob)
        return model

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    torch.cuda.synchronize()
    ts = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - ts

    # second timed region: the same steps with per-launch events
    fb.timing_enable(("histogram", "apply"))
    torch.cuda.synchronize()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    h_launches, h_ms, h_bytes = fb.timing_read("histogram")
    a_launches, a_ms, _ = fb.timing_read("apply")
    fb.timing_enable(())

    ms_per_step = elapsed * 1e3 / args.steps
    value = n * d * D * T / (ms_per_step / 1e3)
    hist_avg_ms = h_ms / max(h_launches, 1)
    hist_avg_bytes = h_bytes / max(h_launches, 1)
    achieved = hist_avg_bytes / (hist_avg_ms / 1e3) / 1e9
    apply_events_per_s = n * a_launches / (a_ms / 1e3) if a_ms > 0 else None

    phases = measure_hist_phases(fb, torch, codes, y, spec) if args.phases else None
    if phases:
        print(f"# histogram phases: {json.dumps(phases)}", file=sys.stderr, flush=True)

    # CPU oracle on a bounded sample of the same workload (first trees, all events)
    from oracle import fbdt_oracle as O
    _, xb = O.bin_features(ds["x"], B)
    cpu_T = max(1, args.cpu_trees)
    tc = time.perf_counter()
    O.fit(xb, ds["y"], ds["v"], D, cpu_T, spec.shrinkage, spec.subsample, spec.fit_seed, B)
    cpu_s = time.perf_counter() - tc
    cpu_value = n * d * D * cpu_T / cpu_s

    fits = {}
    for c in filter(None, str(args.fit_workloads).split(",")):
        fits[f"workload{int(c)}"] = measure_fit_workload(int(c), fb, torch)
        print(f"# fit workload {c}: {fits[f'workload{int(c)}']['fit_ms']:.1f} ms", file=sys.stderr,
              flush=True)

    section4 = measure_section4(fb, torch) if args.section4 else None
    if section4:
        print(f"# section 4 features: {section4}", file=sys.stderr, flush=True)

    apply_out = {"events_per_s": apply_events_per_s, "launches": a_launches,
                 "mean_launch_us": a_ms * 1e3 / max(a_launches, 1),
                 "workload": f"{n} binned events x {T} trees of depth {D} (the step's apply)"}
    if apply_x:
        apply_out = measure_apply_workload(args, apply_x, fb, torch)

    oracle_model = apply_out.pop("_oracle_model", None)
    oracle_baseline = measure_oracle_baseline(oracle_model) if args.oracle_baseline else None

    if args.copy_calibration_mib > 0:
        nbytes = args.copy_calibration_mib << 20
        src = torch.empty(nbytes, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()

    out = {
        "metric": METRIC,
        "value": value,
        "unit": "event*features/s per tree layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {
            "workload": "fit 500k x 20 float32 features, 256 equal-frequency bins, depth 3, "
                        "100 trees, shrinkage 0.1, subsample 0.5 (Gaussian signal/background, "
                        "mean shifts 0.1-0.5 on 10 features) + apply of the fitted forest to "
                        "the 500k binned events",
            "n_events": n, "n_features": d, "n_bins": B, "depth": D, "n_trees": T,
            "histogram_layout": "masked streaming, uint8 feature-major codes",
            "dataset_sha256": digest(ds["x"], ds["y"]),
        },
        "roofline": {
            "bound": "hbm",
            "kernel": "hist_kernel (per-layer histogram with fused routing)",
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS,
            "traffic": measured_traffic(),
            "launches": h_launches,
            "mean_launch_us": hist_avg_ms * 1e3,
            "algorithmic_bytes_per_launch": hist_avg_bytes,
        },
        "hist_phases": phases,
        "apply": apply_out,
        "fit_workloads": fits,
        "section4": section4,
        "bin_ms": bin_ms,
        "bin_warm_ms": bin_warm_ms,
        "oracle_baseline": oracle_baseline,
        "cpu_baseline": {
            "value": cpu_value,
            "unit": "event*features/s per tree layer",
            "cores": 1,
            "host": host_info(),
            "kind": "oracle",
            "sample": f"numpy oracle fit of the first {cpu_T} of the 100 trees on all 500k "
                      f"events (bins precomputed), {cpu_s:.1f} s",
        },
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
