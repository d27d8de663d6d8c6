"""Parity at the full tree counts of the 2M x 40 (200 trees), 10M x 40
(depth 6, 100 trees) and 400-tree workloads, against fits of the CPU oracle
stored by tests/golden/make_full_fixtures.py (the oracle takes 13 to 75
minutes for them, too long to rerun here).

Compared:
  boundaries exactly, the bin codes through the SHA-256 of the oracle's;
  every cut (feature, bin) of every tree exactly; at the first cut that
  differs, the GPU's cut must be in the oracle's near-tie set of that node
  (stored with the fixture), else the test fails naming the node; after such
  an adoption the oracle is resumed at that tree from the scores its own
  earlier trees give (apply of the stored trees, which reproduces the loop's
  scores exactly) with the GPU's cuts as the reference, and the remaining
  trees are compared like the others;
  f0 to 1e-12, boost weights and gains to relative 1e-9 (float64 sums in
  another order), the final score F on the stored event subset to relative
  1e-9, and P of fbdt_apply on that subset to |dP| <= 1e-5.
The 400-tree forest is then applied at the launch shape of the 50M-event
workload to 1.2M fresh events: every event's F equals the oracle's apply of
the same forest, and P is within 1e-5 of it and of the oracle's own forest.
"""
import hashlib
import os
import time

import numpy as np
import pytest
import torch

import paper_1609_06119_amd as fb
from oracle import fbdt_oracle as O
from synth import CONFIGS, make_apply_chunk, make_training_set
from oracle_pool import bin_features_parallel

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
CASES = ["config3-T200", "config4-T100", "config5-T400"]
# oracle seconds per tree on one host core (measured while writing the
# fixtures), to bound a resumed comparison
ORACLE_S_PER_TREE = {"config3-T200": 3.8, "config4-T100": 68.0, "config5-T400": 3.9}
RESUME_BUDGET_S = 420.0


def say(msg):
    print(msg, flush=True)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


@pytest.fixture(autouse=True)
def _defaults():
    for name in ("hist_features_per_group", "hist_event_chunks", "hist_threads", "hist_copies",
                 "apply_threads"):
        fb.set_option(name, 0)
    fb.set_option("fit_graphs", 1)
    yield


def _fixture(case):
    path = os.path.join(GOLDEN, f"full_{case}.npz")
    if not os.path.exists(path):
        pytest.fail(f"{path} is missing (python tests/golden/make_full_fixtures.py {case})")
    with np.load(path, allow_pickle=False) as z:
        return {k: z[k] for k in z.files}


def _near_ties(fx):
    """{(tree, heap node): {(feature, cut): gain}} of the stored near-tie sets."""
    out, k = {}, 0
    for t, node, cnt in fx["nt_node"]:
        out[(int(t), int(node))] = {
            (int(fx["nt_feature"][k + i]), int(fx["nt_cut"][k + i])): float(fx["nt_gain"][k + i])
            for i in range(int(cnt))}
        k += int(cnt)
    return out


def _first_mismatch(gf, gc, of, oc):
    diff = np.argwhere((gf != of) | (gc != oc))
    if diff.size == 0:
        return None
    t = int(diff[:, 0].min())
    k = int(diff[diff[:, 0] == t][:, 1].min())
    return t, k + 1


def _oracle_model(fx, T=None):
    T = int(fx["n_trees"]) if T is None else T
    return O.Model(int(fx["depth"]), int(fx["n_bins"]), int(fx["d"]), float(fx["f0"]),
                   fx["cut_feature"][:T], fx["cut_bin"][:T], fx["gain"][:T], fx["leaf"][:T])


def _fit_and_compare(case):
    fx = _fixture(case)
    spec = CONFIGS[int(fx["fit_workload"])]
    B, D, T = int(fx["n_bins"]), int(fx["depth"]), int(fx["n_trees"])
    assert (B, D, T) == (spec.n_bins, spec.depth, spec.n_trees)
    ds = make_training_set(int(fx["data_workload"]))
    d, n = ds["x"].shape
    assert (n, d) == (int(fx["n"]), int(fx["d"]))
    say(f"fixture parity {case}: n={n} d={d} B={B} D={D} T={T}")
    bounds, codes = fb.bin(dev(ds["x"]), B)
    assert np.array_equal(bounds, fx["boundaries"])
    digest = hashlib.sha256(np.ascontiguousarray(codes.numpy()).tobytes()).hexdigest()
    assert digest == str(fx["codes_sha256"])
    score = torch.empty(n, dtype=torch.float64, device="cuda")
    t0 = time.time()
    model = fb.fit(codes, dev(ds["y"]), B, D, T, float(fx["shrinkage"]), float(fx["subsample"]),
                   int(fx["seed"]), score_out=score)
    gm = model.export()
    say(f"  GPU fit {time.time() - t0:.2f}s")
    of, oc = fx["cut_feature"].copy(), fx["cut_bin"].copy()
    oleaf, ogain = fx["leaf"].copy(), fx["gain"].copy()
    idx = fx["sample_index"]
    oF = fx["sample_F"]
    adopted = []
    mm = _first_mismatch(gm["cut_feature"], gm["cut_bin"], of, oc)
    if mm is not None:
        t, node = mm
        g = (int(gm["cut_feature"][t, node - 1]), int(gm["cut_bin"][t, node - 1]))
        o = (int(of[t, node - 1]), int(oc[t, node - 1]))
        ties = _near_ties(fx).get((t, node), {})
        assert g in ties, (f"{case}: tree {t} node {node}: GPU cut {g}, oracle cut {o} "
                           f"(gain {float(ogain[t, node - 1])!r}); not a near-tie")
        need = (T - t) * ORACLE_S_PER_TREE[case]
        assert need <= RESUME_BUDGET_S, (
            f"{case}: near-tie at tree {t} node {node} (GPU {g}, oracle {o}); the remaining "
            f"{T - t} trees need ~{need:.0f}s of oracle time, over this test's budget")
        say(f"  near-tie at tree {t} node {node}: GPU {g}, oracle {o}; resuming the oracle")
        _, xb = bin_features_parallel(ds["x"], B)
        _, Ft = O.apply(_oracle_model(fx, t), xb)
        ref = O.Model(D, B, d, gm["f0"], gm["cut_feature"], gm["cut_bin"], gm["gain"], gm["leaf"])
        log = O.TieLog()
        om, F = O.fit(xb, ds["y"], ds["v"], D, T, float(fx["shrinkage"]), float(fx["subsample"]),
                      int(fx["seed"]), B, reference=ref, tie_log=log, final_score=True,
                      start=(t, Ft))
        assert log.rejected == [], f"{case}: cuts differ after the resumed tree: {log.rejected[:3]}"
        adopted = log.adopted
        of[t:], oc[t:] = om.cut_feature[t:], om.cut_bin[t:]
        oleaf[t:], ogain[t:] = om.leaf[t:], om.gain[t:]
        oF = F[idx]
    say(f"  near-ties adopted: {len(adopted) + (mm is not None)}")
    assert np.array_equal(gm["cut_feature"], of)
    assert np.array_equal(gm["cut_bin"], oc)
    assert abs(gm["f0"] - float(fx["f0"])) <= 1e-12
    assert np.allclose(gm["leaf"], oleaf, rtol=1e-9, atol=1e-13)
    assert np.allclose(gm["gain"], ogain, rtol=1e-9, atol=1e-12 * n)
    Fg = score.cpu().numpy()[idx]
    assert np.allclose(Fg, oF, rtol=1e-9, atol=1e-12)
    p = fb.apply(model, codes).cpu().numpy()[idx]
    if mm is None:
        assert np.max(np.abs(p.astype(np.float64) - fx["sample_P"])) <= 1e-5
    return fx, model, bounds


@pytest.mark.parametrize("case", ["config3-T200", "config4-T100"])
def test_full_tree_count_fit_matches_oracle_fixture(case):
    _fit_and_compare(case)


def test_400_tree_forest_fit_and_apply_at_the_50M_launch_shape():
    fx, model, bounds = _fit_and_compare("config5-T400")
    d = int(fx["d"])
    n = 1_200_003          # every n >= 524k events takes the grid of the 50M launch
    say(f"  apply of the fitted 400-tree forest to {n} fresh events")
    x = make_apply_chunk(11, n)["x"]
    ob = fx["boundaries"]
    codes = fb.bin_transform(dev(x), bounds)
    xb = np.stack([O.encode(x[j], ob[j]) for j in range(d)]).astype(np.uint8)
    assert np.array_equal(codes.numpy(), xb)
    score = torch.empty(n, dtype=torch.float64, device="cuda")
    p = fb.apply(model, codes, score=score).cpu().numpy().astype(np.float64)
    gm = model.export()
    mine = O.Model(int(fx["depth"]), int(fx["n_bins"]), d, gm["f0"], gm["cut_feature"],
                   gm["cut_bin"], gm["gain"], gm["leaf"])
    say("  oracle apply of the same forest")
    op, oF = O.apply(mine, xb)
    assert np.array_equal(score.cpu().numpy(), oF)
    assert np.max(np.abs(p - op)) <= 1e-5
    say("  oracle apply of the oracle's own forest")
    op2, _ = O.apply(_oracle_model(fx), xb)
    assert np.max(np.abs(p - op2)) <= 1e-5
