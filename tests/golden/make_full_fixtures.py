"""Writes the oracle's fits of the full-size workloads at their full tree
counts as fixtures for the GPU parity tests (tests/test_gpu_fixtures.py).

Run on a CPU (tens of minutes for the 10M-event workload):

    python tests/golden/make_full_fixtures.py [case ...]

Cases (default: all):
  config3-T200   2M x 40, 256 bins, depth 3, 200 trees (fit seed 2)
  config4-T100   10M x 40 mixed marginals, 256 bins, depth 6, 100 trees (fit seed 3)
  config5-T400   the 400-tree depth-3 forest on the 2M x 40 sample (fit seed 4)

Everything stored comes from the CPU oracle (``oracle/fbdt_oracle.py``) on
the seeded synthetic inputs of ``synth/``; nothing here touches the GPU
library.  The binning runs feature by feature in worker processes through
the oracle's own functions (``tests/oracle_pool.py``); the fit is the
oracle's single-threaded loop.  Each fixture (``full_<case>.npz``, no
pickled objects) holds:
  the hyper-parameters and the SHA-256 of the oracle's bin codes;
  the boundaries [d][B-1];
  f0, cut_feature, cut_bin, gain [T][2^D-1] and leaf [T][2^D] (times eta);
  the near-tie sets of the nodes where more than the best cut passes the
  near-tie rule (``nt_*``: tree, heap node, then (feature, cut, gain) rows);
  the final score F and P = apply's probability on a strided subset of the
  events (every ``stride``-th event plus the last one).
"""
from __future__ import annotations

import hashlib
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
for p in (ROOT, os.path.join(ROOT, "tests")):
    if p not in sys.path:
        sys.path.insert(0, p)

from oracle import fbdt_oracle as O  # noqa: E402
from oracle_pool import bin_features_parallel  # noqa: E402
from synth import CONFIGS, make_training_set  # noqa: E402

# case -> (data workload, spec whose fit parameters are used)
CASES = {
    "config3-T200": (3, 3),
    "config4-T100": (4, 4),
    "config5-T400": (3, 5),
}
SAMPLE_EVENTS = 20_000


def codes_digest(xb) -> str:
    return hashlib.sha256(np.ascontiguousarray(xb, dtype=np.uint8).tobytes()).hexdigest()


def sample_index(n: int) -> np.ndarray:
    stride = max(1, n // SAMPLE_EVENTS)
    idx = np.arange(0, n, stride, dtype=np.int64)
    return idx if idx[-1] == n - 1 else np.append(idx, n - 1)


def make(case: str) -> str:
    data_cfg, fit_cfg = CASES[case]
    spec = CONFIGS[fit_cfg]
    B, D, T = spec.n_bins, spec.depth, spec.n_trees
    t0 = time.time()
    ds = make_training_set(data_cfg)
    d, n = ds["x"].shape
    bounds, xb = bin_features_parallel(ds["x"], B, workers=8)
    del ds["x"]
    print(f"{case}: n={n} d={d} binned in {time.time() - t0:.0f}s", flush=True)
    t1 = time.time()
    near = []
    model, F = O.fit(xb, ds["y"], ds["v"], D, T, spec.shrinkage, spec.subsample, spec.fit_seed,
                     B, final_score=True, near_ties=near)
    print(f"{case}: fit of {T} trees in {time.time() - t1:.0f}s, "
          f"{len(near)} nodes with near-ties", flush=True)
    idx = sample_index(n)
    P, Fa = O.apply(model, xb[:, idx])
    nt_rows = [(t, node, len(c)) for t, node, c in near]
    nt_cand = [row for _, _, c in near for row in c]
    out = os.path.join(HERE, f"full_{case}.npz")
    np.savez_compressed(
        out,
        data_workload=np.int64(data_cfg), fit_workload=np.int64(fit_cfg),
        n=np.int64(n), d=np.int64(d), n_bins=np.int64(B), depth=np.int64(D),
        n_trees=np.int64(T), shrinkage=np.float64(spec.shrinkage),
        subsample=np.float64(spec.subsample), seed=np.int64(spec.fit_seed),
        codes_sha256=np.array(codes_digest(xb)), boundaries=bounds,
        f0=np.float64(model.f0), cut_feature=model.cut_feature, cut_bin=model.cut_bin,
        gain=model.gain, leaf=model.leaf,
        nt_node=np.array(nt_rows, np.int64).reshape(-1, 3),
        nt_feature=np.array([r[0] for r in nt_cand], np.int64),
        nt_cut=np.array([r[1] for r in nt_cand], np.int64),
        nt_gain=np.array([r[2] for r in nt_cand], np.float64),
        sample_index=idx, sample_F=F[idx], sample_apply_F=Fa, sample_P=P)
    print(f"{case}: wrote {out} ({os.path.getsize(out)} bytes) in {time.time() - t0:.0f}s",
          flush=True)
    return out


if __name__ == "__main__":
    for c in sys.argv[1:] or list(CASES):
        make(c)
