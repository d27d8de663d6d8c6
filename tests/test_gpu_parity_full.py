"""Parity at the full sizes of the 2M x 40 and 10M x 40 workloads.

The GPU fits the first trees of each workload at its full event count,
feature count, bin count and depth, so every launch has the shape of the
full fit's (launch shapes depend on the events, features, bins and layer,
not on the number of trees); the oracle fits the same trees.  Tolerances are
those of the other parity tests: bin codes, boundaries and tree structure
exact (near-ties of the oracle's gains adopted and counted), boost weights,
gains and scores to relative 1e-9, probabilities to |dP| <= 1e-5.  The
oracle bins the features in spawned worker processes (its own functions,
one feature per task); everything else runs single-threaded.
"""
import numpy as np
import pytest
import torch

import paper_1609_06119_amd as fb
from oracle import fbdt_oracle as O
from synth import CONFIGS, make_training_set
from oracle_pool import bin_features_parallel

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


def say(msg):
    print(msg, flush=True)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


@pytest.fixture(autouse=True)
def _defaults():
    for name in ("hist_features_per_group", "hist_event_chunks", "hist_threads", "hist_copies"):
        fb.set_option(name, 0)
    fb.set_option("fit_graphs", 1)
    yield


FULL_CASES = {
    "config3-2Mx40-20trees": dict(cfg=3, n_trees=20),
    "config4-10Mx40-D6-3trees": dict(cfg=4, n_trees=3),
}


@pytest.mark.parametrize("case", list(FULL_CASES))
def test_full_size_fit_matches_oracle(case):
    c = FULL_CASES[case]
    spec = CONFIGS[c["cfg"]]
    T, B, D = c["n_trees"], spec.n_bins, spec.depth
    ds = make_training_set(c["cfg"])
    d, n = ds["x"].shape
    assert n == spec.n_events and d == spec.n_features
    say(f"full-size parity {case}: n={n} d={d} B={B} D={D} T={T}")
    ob, xb = bin_features_parallel(ds["x"], B)
    bounds, codes = fb.bin(dev(ds["x"]), B)
    assert np.array_equal(bounds, ob)
    assert np.array_equal(codes.numpy(), xb)
    del ds["x"]
    score = torch.empty(n, dtype=torch.float64, device="cuda")
    model = fb.fit(codes, dev(ds["y"]), B, D, T, spec.shrinkage, spec.subsample, spec.fit_seed,
                   score_out=score)
    gm = model.export()
    say(f"  oracle fit {case}")
    ref = O.Model(gm["depth"], gm["n_bins"], gm["n_features"], gm["f0"], gm["cut_feature"],
                  gm["cut_bin"], gm["gain"], gm["leaf"])
    log = O.TieLog()
    om, F = O.fit(xb, ds["y"], ds["v"], D, T, spec.shrinkage, spec.subsample, spec.fit_seed, B,
                  reference=ref, tie_log=log, final_score=True)
    say(f"  near-ties adopted: {len(log.adopted)}  rejected: {len(log.rejected)}")
    assert log.rejected == []
    assert np.array_equal(gm["cut_feature"], om.cut_feature)
    assert np.array_equal(gm["cut_bin"], om.cut_bin)
    assert abs(gm["f0"] - om.f0) <= 1e-12
    assert np.allclose(gm["leaf"], om.leaf, rtol=1e-9, atol=1e-13)
    assert np.allclose(gm["gain"], om.gain, rtol=1e-9, atol=1e-12 * n)
    Fg = score.cpu().numpy()
    assert np.allclose(Fg, F, rtol=1e-9, atol=1e-12)
    say(f"  apply {case}")
    p = fb.apply(model, codes).cpu().numpy()
    op, _ = O.apply(om, xb)
    assert np.max(np.abs(p.astype(np.float64) - op)) <= 1e-5
