"""Parity of the HIP library (through its C ABI) with the CPU oracle.

Tolerances: bin codes, boundaries, sub-sample masks, node ids, cut features
and cut bins are compared exactly (tree structure only up to near-ties of
the oracle's gains, relative 1e-6, adopted and counted); histogram sums to
relative 1e-5 (also checked at 1e-12, the float64 accumulation level);
probabilities to |dP| <= 1e-5; scores, gains and boost weights to relative
1e-9 (float64 sums taken in a different order).
"""
import numpy as np
import pytest
import torch

import paper_1609_06119_amd as fb
from oracle import fbdt_oracle as O
from synth import CONFIGS, make_apply_chunk, make_training_set, random_forest

pytestmark = pytest.mark.gpu

HIST_RTOL = 1e-5


def say(msg):
    print(msg, flush=True)


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def max_rel(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    den = np.maximum(np.abs(b), 1e-300)
    return float(np.max(np.where(a == b, 0.0, np.abs(a - b) / den))) if a.size else 0.0


@pytest.fixture(autouse=True)
def _defaults():
    for name in ("hist_features_per_group", "hist_event_chunks", "hist_threads",
                 "hist_copies", "apply_threads"):
        fb.set_option(name, 0)
    fb.set_option("fit_graphs", 1)
    yield
    for name in ("hist_features_per_group", "hist_event_chunks", "hist_threads",
                 "hist_copies", "apply_threads"):
        fb.set_option(name, 0)
    fb.set_option("fit_graphs", 1)


# ------------------------------------------------------------------ binning
def _bin_cases():
    rng = np.random.default_rng(0)
    cases = [("config1", make_training_set(1)["x"], 16),
             ("config2-100k", make_training_set(2, n_events=100_003)["x"], 256),
             ("config4-50k", make_training_set(4, n_events=50_001)["x"], 256)]
    x = rng.normal(size=(3, 1001)).astype(np.float32)
    x[0, :10] = np.inf
    x[1, :10] = -np.inf
    x[2, ::3] = 0.0
    x[2, 1::3] = -0.0
    cases.append(("inf-and-signed-zero", x, 32))
    cases.append(("one-event", np.array([[1.5]], np.float32), 2))
    cases.append(("more-bins-than-events", rng.normal(size=(2, 5)).astype(np.float32), 256))
    # subnormal, tiny, huge and signed-zero values mixed (the order-preserving
    # keys of the device sort against the oracle's comparison sort)
    edge = np.array([1e-45, -1e-45, 1e-40, -1e-40, 1.17549435e-38, 0.0, -0.0, 3.4028235e38,
                     -3.4028235e38, 1.0, -1.0], np.float32)
    cases.append(("subnormal-and-huge", edge[rng.integers(0, len(edge), (3, 4001))], 64))
    return cases


@pytest.mark.parametrize("case", range(7))
def test_bin_matches_oracle(case):
    name, x, B = _bin_cases()[case]
    say(f"bin parity: {name} d={x.shape[0]} n={x.shape[1]} B={B}")
    d, n = x.shape
    # binning writes the first n codes of each row only: padding keeps its bytes
    pre = torch.full((d, fb.padded_stride(n)), 0xAB, dtype=torch.uint8, device="cuda")
    bounds, codes = fb.bin(dev(x), B, codes=fb.Codes(pre, n))
    ob, oc = O.bin_features(x, B)
    assert np.array_equal(bounds, ob)
    assert np.array_equal(codes.numpy(), oc)
    pad = codes.data[:, codes.n:].cpu().numpy()
    assert (pad == 0xAB).all()


def test_bin_with_row_stride_and_transform():
    ds = make_training_set(1)
    x = ds["x"]
    wide = np.zeros((x.shape[0], x.shape[1] + 37), np.float32)
    wide[:, : x.shape[1]] = x
    xw = dev(wide)[:, : x.shape[1]]
    say("bin with ldx > n")
    bounds, codes = fb.bin(xw, 16)
    ob, oc = O.bin_features(x, 16)
    assert np.array_equal(bounds, ob) and np.array_equal(codes.numpy(), oc)
    fresh = make_apply_chunk(0, 30_001)["x"][:8]
    say("bin_transform of fresh events")
    c2 = fb.bin_transform(dev(fresh), bounds)
    ref = np.stack([O.encode(fresh[j], ob[j]) for j in range(8)])
    assert np.array_equal(c2.numpy(), ref)


def test_bin_rejects_nan_with_256_bins():
    """NaN takes the reserved code 255 (section 4.2), so it is an error only
    when all 256 codes are bins."""
    x = np.ones((2, 100), np.float32)
    x[1, 50] = np.nan
    with pytest.raises(fb.FbdtError) as ei:
        fb.bin(dev(x), 256)
    assert ei.value.status == "FBDT_E_NAN"
    with pytest.raises(fb.FbdtError) as ei:
        fb.bin_transform(dev(x), np.zeros((2, 255), np.float32))
    assert ei.value.status == "FBDT_E_NAN"


def _with_missing(x, seed):
    """A copy of x [d][n] with NaN values (section 4.2): features in turn
    hold none, 3 %, 20 % and 60 % NaN; the last feature is NaN throughout."""
    rng = np.random.default_rng(seed)
    x = np.array(x, np.float32)
    d, n = x.shape
    for j in range(d):
        frac = (0.0, 0.03, 0.2, 0.6)[j % 4]
        x[j, rng.random(n) < frac] = np.nan
    x[d - 1] = np.nan
    return x


@pytest.mark.parametrize("cfg,n,B", [(1, None, 16), (4, 50_001, 255), (2, 30_011, 2)])
def test_bin_with_missing_values_matches_oracle(cfg, n, B):
    x = _with_missing(make_training_set(cfg, n_events=n)["x"], cfg)
    x[0, :5] = -np.nan                                  # a NaN with the sign bit set
    say(f"bin with NaN: workload {cfg} d={x.shape[0]} n={x.shape[1]} B={B}")
    bounds, codes = fb.bin(dev(x), B)
    ob, oc = O.bin_features(x, B)
    assert np.array_equal(bounds, ob)
    assert np.array_equal(codes.numpy(), oc)
    assert np.isinf(bounds[-1]).all() and (oc[-1] == O.MISSING).all()
    fresh = _with_missing(make_apply_chunk(1, 20_001)["x"][: x.shape[0]], 99)
    c2 = fb.bin_transform(dev(fresh), bounds)
    ref = np.stack([O.encode(fresh[j], ob[j]) for j in range(x.shape[0])])
    assert np.array_equal(c2.numpy(), ref)


# ------------------------------------------------------------ single steps
def test_tree_weights_match_oracle():
    rng = np.random.default_rng(1)
    n = 100_003
    y = np.where(rng.random(n) < 0.5, 1, -1).astype(np.int8)
    v = rng.uniform(0, 2, n).astype(np.float32)
    v[:100] = 0
    F = rng.normal(0, 2, n)
    for tree, alpha in ((0, 0.5), (7, 0.3), (2, 1.0)):
        say(f"tree_weights tree={tree} alpha={alpha}")
        w = fb.tree_weights(dev(y), dev(v), dev(F), seed=99, tree=tree, alpha=alpha).cpu().numpy()
        mask = O.subsample_mask(99, tree, n, alpha)
        ow = O.histogram_weights(y, v, O.pseudo_response(y, F), mask)
        ows = np.where(y > 0, ow, -ow).astype(np.float32)
        assert np.array_equal(w != 0, ows != 0)
        assert np.array_equal(np.signbit(w[w != 0]), np.signbit(ows[ows != 0]))
        np.testing.assert_array_max_ulp(w, ows, maxulp=1)
        if alpha < 1.0:
            sampled = (w != 0) | (v == 0) & mask
            assert np.array_equal(sampled[v != 0], mask[v != 0])


@pytest.mark.parametrize("layer,n_bins,d,n", [(0, 256, 7, 65_539), (1, 16, 3, 1000),
                                              (2, 256, 20, 100_001), (3, 64, 5, 20_000),
                                              (5, 256, 4, 50_003), (6, 256, 2, 30_001),
                                              (0, 2, 1, 1), (4, 256, 9, 7)])
def test_histogram_matches_oracle(layer, n_bins, d, n):
    rng = np.random.default_rng(layer * 31 + n_bins)
    xb = rng.integers(0, n_bins, (d, n)).astype(np.uint8)
    node = rng.integers(1 << layer, 2 << layer, n).astype(np.uint8)
    y = np.where(rng.random(n) < 0.45, 1, -1).astype(np.int8)
    wa = rng.uniform(0, 2, n).astype(np.float32)
    wa[rng.random(n) < 0.5] = 0
    ws = np.where(y > 0, wa, -wa).astype(np.float32)
    ref = O.histogram(xb, node.astype(np.int64), wa, y > 0, layer, n_bins)
    codes = fb.Codes.from_numpy(xb)
    for chunks in (0, 1, 3, 17):
        fb.set_option("hist_event_chunks", chunks)
        say(f"histogram layer={layer} B={n_bins} d={d} n={n} chunks={chunks}")
        H = fb.histogram(codes, dev(node), dev(ws), layer, n_bins).cpu().numpy()
        assert np.array_equal(H == 0, ref == 0)
        err = max_rel(H, ref)
        assert err <= HIST_RTOL
        assert err <= 1e-12, err


@pytest.mark.parametrize("layer", [0, 3])
def test_histogram_weights_of_every_magnitude(layer):
    # weights from 1e-12 to 1e3: the large ones are summed exactly in fixed
    # point, the ones below the fixed-point grid in float64
    rng = np.random.default_rng(11 + layer)
    n, d, B = 60_013, 5, 64
    xb = rng.integers(0, B, (d, n)).astype(np.uint8)
    node = rng.integers(1 << layer, 2 << layer, n).astype(np.uint8)
    y = np.where(rng.random(n) < 0.5, 1, -1).astype(np.int8)
    wa = (10.0 ** rng.uniform(-12, 3, n)).astype(np.float32)
    wa[rng.random(n) < 0.3] = 0
    ws = np.where(y > 0, wa, -wa).astype(np.float32)
    ref = O.histogram(xb, node.astype(np.int64), wa, y > 0, layer, B)
    say(f"histogram weights 1e-12..1e3 layer={layer}")
    H = fb.histogram(fb.Codes.from_numpy(xb), dev(node), dev(ws), layer, B).cpu().numpy()
    assert np.array_equal(H == 0, ref == 0)
    assert max_rel(H, ref) <= 1e-12


def test_histogram_feature_groups_and_threads():
    rng = np.random.default_rng(3)
    n, d, B, layer = 40_001, 11, 256, 2
    xb = rng.integers(0, B, (d, n)).astype(np.uint8)
    node = rng.integers(4, 8, n).astype(np.uint8)
    y = np.where(rng.random(n) < 0.5, 1, -1).astype(np.int8)
    wa = rng.uniform(0.1, 1, n).astype(np.float32)
    ws = np.where(y > 0, wa, -wa).astype(np.float32)
    ref = O.histogram(xb, node.astype(np.int64), wa, y > 0, layer, B)
    codes = fb.Codes.from_numpy(xb)
    for fpg, threads, copies in ((2, 256, 4), (4, 512, 2), (5, 1024, 1), (8, 128, 4), (1, 64, 2),
                                 (5, 1024, 4)):
        fb.set_option("hist_features_per_group", fpg)
        fb.set_option("hist_threads", threads)
        fb.set_option("hist_copies", copies)
        say(f"histogram fpg={fpg} threads={threads} copies={copies}")
        H = fb.histogram(codes, dev(node), dev(ws), layer, B).cpu().numpy()
        assert max_rel(H, ref) <= 1e-12


def test_histogram_copies_with_few_distinct_codes():
    """Every lane of an instruction hitting the same few counters (a feature
    with two codes) is summed exactly with one, two or four LDS copies."""
    rng = np.random.default_rng(4)
    n, d, B, layer = 70_003, 5, 256, 1
    xb = rng.integers(0, 2, (d, n)).astype(np.uint8) * 255
    node = rng.integers(2, 4, n).astype(np.uint8)
    y = np.where(rng.random(n) < 0.5, 1, -1).astype(np.int8)
    wa = rng.uniform(0.1, 1, n).astype(np.float32)
    ws = np.where(y > 0, wa, -wa).astype(np.float32)
    ref = O.histogram(xb, node.astype(np.int64), wa, y > 0, layer, B)
    codes = fb.Codes.from_numpy(xb)
    for copies in (1, 2, 4):
        fb.set_option("hist_copies", copies)
        H = fb.histogram(codes, dev(node), dev(ws), layer, B).cpu().numpy()
        assert max_rel(H, ref) <= 1e-12


def _check_cuts(H, f, c, g):
    S, Bk = O.cumulative(H)
    gains = O.split_gains(S, Bk)
    of, oc, og = O.best_cuts(gains)
    n_bins = H.shape[2]
    parent = O.gini(S[:, 0, n_bins], Bk[:, 0, n_bins])
    ties = 0
    for k in range(H.shape[0]):
        if (f[k], c[k]) != (of[k], oc[k]):
            other = gains[k, f[k], c[k] - 1]
            assert O.is_near_tie(og[k], other, parent[k]), (k, (f[k], c[k]), (of[k], oc[k]))
            ties += 1
        assert abs(g[k] - gains[k, f[k], c[k] - 1]) <= 1e-12 * max(abs(parent[k]), 1e-300)
    return ties


@pytest.mark.parametrize("seed", range(6))
def test_best_cuts_match_oracle(seed):
    rng = np.random.default_rng(seed)
    n_nodes = [1, 2, 4, 8, 32, 64][seed]
    d = [1, 3, 5, 20, 7, 2][seed]
    B = [2, 16, 256, 256, 64, 256][seed]
    H = rng.uniform(0, 5, (n_nodes, d, B, 2))
    H[rng.random(H.shape) < 0.3] = 0.0              # empty bins
    if n_nodes > 1:
        H[1] = 0.0                                   # an empty node
        H[0, :, :, 1] = 0.0                          # a pure node
    say(f"best_cuts nodes={n_nodes} d={d} B={B}")
    f, c, g = (t.cpu().numpy() for t in fb.best_cuts(dev(H)))
    _check_cuts(H, f, c, g)
    if n_nodes > 1:
        assert (f[1], c[1], g[1]) == (0, 1, 0.0)
        assert (f[0], c[0], g[0]) == (0, 1, 0.0)


def test_best_cuts_exact_ties_take_lowest_feature_and_bin():
    # XOR root (Table 3, section 4.3): every gain is exactly 0
    H = np.zeros((1, 2, 2, 2))
    H[0, :, :, :] = 1.0
    f, c, g = (t.cpu().numpy() for t in fb.best_cuts(dev(H)))
    assert (f[0], c[0], g[0]) == (0, 1, 0.0)
    # two identical features: the lower wins; duplicate bins: the lower cut wins
    H = np.zeros((1, 3, 8, 2))
    H[0, :, 2, 0] = 3.0
    H[0, :, 6, 1] = 2.0
    H[0, 0, :, :] = 0.0
    H[0, 0, 0, 0] = 5.0
    f, c, g = (t.cpu().numpy() for t in fb.best_cuts(dev(H)))
    assert (f[0], c[0]) == (1, 3)


def test_route_matches_oracle():
    rng = np.random.default_rng(4)
    n, d, B = 70_001, 6, 32
    xb = rng.integers(0, B, (d, n)).astype(np.uint8)
    codes = fb.Codes.from_numpy(xb)
    for layer in (0, 1, 3, 6):
        node = rng.integers(1 << layer, 2 << layer, n).astype(np.uint8)
        cf = rng.integers(0, d, 1 << layer).astype(np.uint8)
        cc = rng.integers(1, B, 1 << layer).astype(np.uint8)
        say(f"route layer={layer}")
        got = fb.route(codes, dev(node), dev(cf), dev(cc), layer).cpu().numpy()
        ref = O.route(node.astype(np.int64), xb, cf, cc, layer)
        assert np.array_equal(got.astype(np.int64), ref)


def test_leaf_values_match_oracle():
    rng = np.random.default_rng(5)
    n = 90_001
    for depth in (1, 3, 6, 7):
        leaf_id = rng.integers(1 << depth, 2 << depth, n).astype(np.uint8)
        leaf_id[leaf_id == (1 << depth) + 1] = 1 << depth     # one empty leaf
        y = np.where(rng.random(n) < 0.5, 1, -1).astype(np.int8)
        v = rng.uniform(0.2, 2, n).astype(np.float32)
        F = rng.normal(0, 1.5, n)
        say(f"leaf_values depth={depth}")
        got = fb.leaf_values(dev(leaf_id), dev(y), dev(v), dev(F), depth, seed=7, tree=3,
                             alpha=0.5, eta=0.1).cpu().numpy()
        mask = O.subsample_mask(7, 3, n, 0.5)
        ref = 0.1 * O.leaf_values(leaf_id.astype(np.int64) - (1 << depth),
                                  O.pseudo_response(y, F), v, mask, 1 << depth)
        assert got[1] == 0.0 and ref[1] == 0.0
        assert max_rel(got, ref) <= 1e-12


# --------------------------------------------------------------- full fit
def _oracle_model(m):
    return O.Model(m["depth"], m["n_bins"], m["n_features"], m["f0"], m["cut_feature"],
                   m["cut_bin"], m["gain"], m["leaf"], m.get("inner"))


FIT_CASES = {
    "config1": dict(cfg=1),
    "config2-full": dict(cfg=2),
    "config3-100k-20trees": dict(cfg=3, n_events=100_000, n_trees=20),
    "config4-200k-3trees": dict(cfg=4, n_events=200_000, n_trees=3),
    "ragged-depth1-B2": dict(cfg=1, n_events=1237, depth=1, n_bins=2, n_trees=5),
    "depth7-B128": dict(cfg=3, n_events=40_013, depth=7, n_bins=128, n_trees=2, subsample=1.0),
    "weighted-alpha0.8": dict(cfg=2, n_events=30_011, n_trees=8, weights=True, subsample=0.8),
    # negative event weights (section 4.1): about a fifth of the events
    "negative-weights": dict(cfg=2, n_events=30_011, n_trees=8, weights="signed"),
    "negative-weights-depth6": dict(cfg=4, n_events=60_013, depth=6, n_trees=2, weights="signed"),
    # tiny samples: fewer events than one step of a pass, most nodes empty
    "two-events-depth3": dict(cfg=1, n_events=2, depth=3, n_trees=3, subsample=1.0),
    "17-events-depth6-B4": dict(cfg=4, n_events=17, depth=6, n_bins=4, n_trees=2),
    "1001-events-depth7-B255": dict(cfg=3, n_events=1001, depth=7, n_bins=255, n_trees=2),
    # event weights over 15 orders of magnitude: the smallest fall below the
    # fixed-point grid into the float64 side histograms inside the fit
    "weights-1e-12-to-1e3": dict(cfg=2, n_events=30_011, n_trees=5, weights="wide"),
    # one signal event in 20,000: F0 = -4.95, extreme pseudo-responses
    "one-signal-in-20000": dict(cfg=1, n_events=20_000, n_trees=5, labels="one-signal"),
}


@pytest.mark.parametrize("case", list(FIT_CASES))
def test_fit_and_apply_match_oracle(case):
    c = FIT_CASES[case]
    spec = CONFIGS[c["cfg"]]
    ds = make_training_set(c["cfg"], n_events=c.get("n_events"))
    n = ds["x"].shape[1]
    B = c.get("n_bins", spec.n_bins)
    D = c.get("depth", spec.depth)
    T = c.get("n_trees", spec.n_trees)
    alpha = c.get("subsample", spec.subsample)
    eta = spec.shrinkage
    seed = spec.fit_seed
    v = ds["v"]
    if c.get("weights") == "signed":
        v = np.random.default_rng(9).uniform(-0.6, 2.5, n).astype(np.float32)
    elif c.get("weights") == "wide":
        v = (10.0 ** np.random.default_rng(9).uniform(-12, 3, n)).astype(np.float32)
    elif c.get("weights"):
        v = np.random.default_rng(9).uniform(0.2, 3.0, n).astype(np.float32)
    if c.get("labels") == "one-signal":
        ds["y"] = np.full(n, -1, np.int8)
        ds["y"][n // 3] = 1
    say(f"fit parity {case}: n={n} d={ds['x'].shape[0]} B={B} D={D} T={T} alpha={alpha}")
    bounds, codes = fb.bin(dev(ds["x"]), B)
    ob, xb = O.bin_features(ds["x"], B)
    assert np.array_equal(codes.numpy(), xb)
    score = torch.empty(n, dtype=torch.float64, device="cuda")
    model = fb.fit(codes, dev(ds["y"]), B, D, T, eta, alpha, seed, w=dev(v), score_out=score)
    gm = model.export()
    say(f"  oracle fit {case}")
    log = O.TieLog()
    om, F = O.fit(xb, ds["y"], v, D, T, eta, alpha, seed, B, reference=_oracle_model(gm),
                  tie_log=log, final_score=True)
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
    ascore = torch.empty(n, dtype=torch.float64, device="cuda")
    p = fb.apply(model, codes, score=ascore).cpu().numpy()
    assert np.array_equal(ascore.cpu().numpy(), Fg)          # apply reproduces the fit's F
    op, oF = O.apply(om, xb)
    assert np.max(np.abs(p.astype(np.float64) - op)) <= 1e-5
    assert np.allclose(ascore.cpu().numpy(), oF, rtol=1e-9, atol=1e-12)


MISSING_CASES = {
    "config1-nan": dict(cfg=1),
    "config2-nan-30k-weighted": dict(cfg=2, n_events=30_011, n_trees=8, n_bins=200,
                                     weights=True),
    "config4-nan-60k-depth6-B255": dict(cfg=4, n_events=60_013, n_bins=255, n_trees=3),
    "nan-depth1-B2": dict(cfg=1, n_events=1237, depth=1, n_bins=2, n_trees=5),
    "nan-negative-weights": dict(cfg=2, n_events=30_011, depth=4, n_trees=4, n_bins=64,
                                 weights="signed"),
    "nan-33-events-depth5": dict(cfg=1, n_events=33, depth=5, n_trees=3),
    "nan-depth7-B64": dict(cfg=2, n_events=40_009, depth=7, n_bins=64, n_trees=3),
}


@pytest.mark.parametrize("case", list(MISSING_CASES))
def test_fit_with_missing_values_matches_oracle(case):
    """Section 4.2: NaN values take the missing code, stay out of their
    feature's histograms, and stop an event at the node that cuts on them;
    every node gets a boost weight.  The fitted model (cuts, gains, leaf and
    inner-node weights), the fit's final scores, and the binned apply, float
    apply and event importance of that model against the oracle."""
    c = MISSING_CASES[case]
    spec = CONFIGS[c["cfg"]]
    ds = make_training_set(c["cfg"], n_events=c.get("n_events"))
    x = _with_missing(ds["x"], 7)
    d, n = x.shape
    B = c.get("n_bins", spec.n_bins)
    D = c.get("depth", spec.depth)
    T = c.get("n_trees", spec.n_trees)
    eta, alpha, seed = spec.shrinkage, spec.subsample, spec.fit_seed
    v = ds["v"]
    if c.get("weights") == "signed":
        v = np.random.default_rng(9).uniform(-0.6, 2.5, n).astype(np.float32)
    elif c.get("weights"):
        v = np.random.default_rng(9).uniform(0.2, 3.0, n).astype(np.float32)
    say(f"missing-value fit {case}: n={n} d={d} B={B} D={D} T={T}")
    bounds, codes = fb.bin(dev(x), B)
    ob, xb = O.bin_features(x, B)
    assert np.array_equal(codes.numpy(), xb)
    score = torch.empty(n, dtype=torch.float64, device="cuda")
    model = fb.fit(codes, dev(ds["y"]), B, D, T, eta, alpha, seed, w=dev(v), score_out=score)
    gm = model.export()
    assert "inner" in gm and gm["inner"].shape == gm["gain"].shape
    say(f"  oracle fit {case}")
    log = O.TieLog()
    om, F = O.fit(xb, ds["y"], v, D, T, eta, alpha, seed, B, reference=_oracle_model(gm),
                  tie_log=log, final_score=True)
    say(f"  near-ties adopted: {len(log.adopted)}  rejected: {len(log.rejected)}")
    assert log.rejected == []
    assert om.inner is not None
    assert np.array_equal(gm["cut_feature"], om.cut_feature)
    assert np.array_equal(gm["cut_bin"], om.cut_bin)
    assert abs(gm["f0"] - om.f0) <= 1e-12
    assert np.allclose(gm["gain"], om.gain, rtol=1e-9, atol=1e-12 * n)
    assert np.allclose(gm["leaf"], om.leaf, rtol=1e-9, atol=1e-13)
    assert np.allclose(gm["inner"], om.inner, rtol=1e-9, atol=1e-13)
    Fg = score.cpu().numpy()
    assert np.allclose(Fg, F, rtol=1e-9, atol=1e-12)
    say(f"  apply {case}")
    ascore = torch.empty(n, dtype=torch.float64, device="cuda")
    p = fb.apply(model, codes, score=ascore).cpu().numpy()
    assert np.array_equal(ascore.cpu().numpy(), Fg)
    op, oF = O.apply(om, xb)
    assert np.max(np.abs(p.astype(np.float64) - op)) <= 1e-5
    assert np.allclose(ascore.cpu().numpy(), oF, rtol=1e-9, atol=1e-12)
    say(f"  apply_float {case}")
    model.set_boundaries(bounds)
    fscore = torch.empty(n, dtype=torch.float64, device="cuda")
    pf = fb.apply_float(model, dev(x), score=fscore).cpu().numpy()
    assert np.array_equal(fscore.cpu().numpy(), Fg)
    assert np.array_equal(pf, p)
    tp, tF = O.apply_thresholds(om, x, ob)
    assert np.array_equal(tF, oF)
    say(f"  event importance {case}")
    ei = fb.event_importance(model, codes).cpu().numpy()
    oe = O.event_importance(om, xb)
    assert np.allclose(ei, oe, rtol=1e-9, atol=1e-12 * n)
    assert np.allclose(fb.feature_importance(model), O.feature_importance(om), rtol=1e-9,
                       atol=1e-12 * n)


def test_plain_data_with_fewer_than_256_bins_stays_plain():
    ds = make_training_set(1)
    y = dev(ds["y"])
    _, plain = fb.bin(dev(ds["x"]), 16)                 # B <= 255 but no NaN
    assert "inner" not in fb.fit(plain, y, 16, 3, 2).export()


@pytest.mark.parametrize("d,n,B,D,T", [(255, 5003, 256, 4, 3), (3, 20_011, 3, 5, 4),
                                       (8, 3001, 16, 2, 300)])
def test_fit_extreme_shapes_match_oracle(d, n, B, D, T):
    """The most features a code byte can name (255), three bins, and a
    300-tree boosting loop (one captured graph of 300 x 6 launches), against
    the oracle: random features, labels from a noisy linear rule."""
    rng = np.random.default_rng(d + n)
    x = rng.normal(size=(d, n)).astype(np.float32)
    score = x[: min(d, 4)].sum(axis=0) + rng.normal(scale=1.0, size=n)
    y = np.where(score > 0, 1, -1).astype(np.int8)
    v = np.ones(n, np.float32)
    say(f"extreme fit: d={d} n={n} B={B} D={D} T={T}")
    _, codes = fb.bin(dev(x), B)
    _, xb = O.bin_features(x, B)
    assert np.array_equal(codes.numpy(), xb)
    sc = torch.empty(n, dtype=torch.float64, device="cuda")
    gm = fb.fit(codes, dev(y), B, D, T, 0.1, 0.5, 3, score_out=sc).export()
    log = O.TieLog()
    om, F = O.fit(xb, y, v, D, T, 0.1, 0.5, 3, B, reference=_oracle_model(gm), tie_log=log,
                  final_score=True)
    say(f"  near-ties adopted: {len(log.adopted)}  rejected: {len(log.rejected)}")
    assert log.rejected == []
    assert np.array_equal(gm["cut_feature"], om.cut_feature)
    assert np.array_equal(gm["cut_bin"], om.cut_bin)
    assert np.allclose(gm["leaf"], om.leaf, rtol=1e-9, atol=1e-13)
    assert np.allclose(sc.cpu().numpy(), F, rtol=1e-9, atol=1e-12)


def test_fit_on_constant_features_takes_zero_gain_cuts():
    """Degenerate sample: every feature constant, so every boundary equals the
    value and every code is the top bin; every candidate cut has gain 0 and
    every node takes (feature 0, bin 1), which sends all its events right:
    only the rightmost leaf has events, the others keep boost weight 0
    (section 1.1's cut rule, the empty-node reading), against the oracle."""
    n, d, B, D, T = 1000, 3, 16, 3, 2
    x = np.full((d, n), 2.5, np.float32)
    y = np.where(np.arange(n) % 3 == 0, 1, -1).astype(np.int8)
    _, codes = fb.bin(dev(x), B)
    _, xb = O.bin_features(x, B)
    assert np.array_equal(codes.numpy(), xb)
    sc = torch.empty(n, dtype=torch.float64, device="cuda")
    gm = fb.fit(codes, dev(y), B, D, T, 0.1, 0.5, 1, score_out=sc).export()
    om, F = O.fit(xb, y, np.ones(n, np.float32), D, T, 0.1, 0.5, 1, B, final_score=True)
    assert (gm["cut_feature"] == 0).all() and (gm["cut_bin"] == 1).all()
    assert np.array_equal(gm["cut_feature"], om.cut_feature)
    assert np.array_equal(gm["cut_bin"], om.cut_bin)
    assert (gm["gain"] == 0.0).all()
    assert np.allclose(gm["leaf"], om.leaf, rtol=1e-12, atol=1e-15)
    assert (gm["leaf"][:, :-1] == 0.0).all()         # only the rightmost leaf has events
    assert np.allclose(sc.cpu().numpy(), F, rtol=1e-12)


@pytest.mark.parametrize("lists", [1, 2], ids=["streaming", "lists"])
def test_fit_on_duplicated_features_keeps_the_first_copy(lists):
    """Every feature followed by an exact copy of itself: each cut on a copy
    has bit for bit the gain of the same cut on the original, so the tie rule
    (highest gain, then lowest feature, section 1.1) must pick the original
    at every node, through the fit's best-cut keys, and the forest must be
    the one fitted on the originals alone (cuts, gains, boost weights and
    scores bit for bit), in the streaming and the list-driven layers."""
    ds = make_training_set(4, n_events=40_009)
    x = ds["x"][:12]
    d, n = x.shape
    B, D, T = 256, 5, 4
    y, v = dev(ds["y"]), dev(ds["v"])
    _, c1 = fb.bin(dev(x), B)
    _, c2 = fb.bin(dev(np.concatenate([x, x])), B)
    assert torch.equal(c2.data[d:2 * d, :n], c1.data[:d, :n])
    fb.set_option("hist_lists", lists)
    try:
        runs = []
        for codes in (c1, c2):
            sc = torch.empty(n, dtype=torch.float64, device="cuda")
            runs.append((fb.fit(codes, y, B, D, T, 0.1, 0.5, 7, w=v, score_out=sc).export(),
                         sc.cpu().numpy()))
    finally:
        fb.set_option("hist_lists", 0)
    (m1, s1), (m2, s2) = runs
    assert (m2["cut_feature"] < d).all()
    for key in ("cut_feature", "cut_bin", "gain", "leaf"):
        assert np.array_equal(m1[key], m2[key]), key
    assert np.array_equal(s1, s2)


@pytest.mark.parametrize("mode", ["plain", "missing-signed-depth5"])
def test_fit_graph_replays_match_eager_fit(mode):
    """The boosting loop is captured once per argument set and replayed; every
    replay, with other device work and other fits in between, gives the model
    and scores of a fit that launches its kernels one by one; also for a fit
    with missing values, negative weights and route passes (depth 5)."""
    spec = CONFIGS[2]
    ds = make_training_set(2, n_events=60_013)
    n = ds["x"].shape[1]
    x, B, D, w = ds["x"], spec.n_bins, 3, None
    if mode != "plain":
        x, B, D = _with_missing(x, 5), 200, 5
        w = dev(np.random.default_rng(9).uniform(-0.6, 2.5, n).astype(np.float32))
    _, codes = fb.bin(dev(x), B)
    y = dev(ds["y"])
    args = (B, D, 12, spec.shrinkage, spec.subsample)

    def run(seed):
        score = torch.empty(n, dtype=torch.float64, device="cuda")
        m = fb.fit(codes, y, *args, seed, w=w, score_out=score).export()
        return m, score.cpu().numpy()

    def same(a, b):
        (ma, fa), (mb, fb_) = a, b
        assert ("inner" in ma) == (mode != "plain") == ("inner" in mb)
        for k in ("cut_feature", "cut_bin", "gain", "leaf") + (("inner",) if "inner" in ma else ()):
            assert np.array_equal(ma[k], mb[k]), k
        assert ma["f0"] == mb["f0"]
        assert np.array_equal(fa, fb_)

    fb.set_option("fit_graphs", 0)
    eager = {s: run(s) for s in (11, 12, 13, 14, 15)}
    fb.set_option("fit_graphs", 1)
    junk = torch.randn(1 << 20, device="cuda")
    for rep in range(3):
        say(f"graph replay {rep}")
        same(run(11), eager[11])
        junk.mul_(1.0001).add_(0.5)             # eager work between replays
        torch.cuda.synchronize()
        same(run(12), eager[12])
    for s in (13, 14, 15, 11):                  # more keys than the cache holds
        same(run(s), eager[s])
    fb.set_option("fit_graphs", 0)              # eager again after replays
    same(run(11), eager[11])


# ------------------------------------------------------------------ apply
@pytest.mark.parametrize("T,D,d,n", [(400, 3, 40, 100_003), (100, 6, 40, 50_001),
                                     (1, 1, 1, 1), (50, 7, 255, 3001), (3, 2, 5, 255)])
def test_apply_random_forest_matches_oracle(T, D, d, n):
    B = 256
    f = random_forest(T, D, d, B, seed=T + D)
    rng = np.random.default_rng(d)
    xb = rng.integers(0, B, (d, n)).astype(np.uint8)
    say(f"apply T={T} D={D} d={d} n={n}")
    model = fb.Model.from_arrays(f["cut_feature"], f["cut_bin"], f["leaf"], f["f0"], d, B)
    codes = fb.Codes.from_numpy(xb)
    score = torch.empty(n, dtype=torch.float64, device="cuda")
    p = fb.apply(model, codes, score=score).cpu().numpy()
    om = O.Model(D, B, d, f["f0"], f["cut_feature"], f["cut_bin"], np.zeros_like(f["leaf"][:, 1:]),
                 f["leaf"])
    op, oF = O.apply(om, xb)
    assert np.array_equal(score.cpu().numpy(), oF)     # same leaves, same order
    assert np.max(np.abs(p.astype(np.float64) - op)) <= 1e-5
    np.testing.assert_array_max_ulp(p, op, maxulp=1)


def test_apply_workload5_launch_configuration_matches_oracle():
    """Workload 5's apply path at its launch configuration (every n >= 524k
    events takes the grid bench.py times on 50M): fresh events from the
    correlated distribution, binned with workload 3's training boundaries on
    both sides, then a seeded 400-tree depth-3 forest over the 40 features;
    all events compared on codes, the first 200k on scores and probabilities."""
    s3, s5 = CONFIGS[3], CONFIGS[5]
    B, D, T = s5.n_bins, s5.depth, s5.n_trees
    say("workload 5: training boundaries (workload 3, 2M x 40)")
    ds = make_training_set(3)
    d = ds["x"].shape[0]
    gb, _ = fb.bin(dev(ds["x"]), B)
    ob = np.stack([O.quantile_boundaries(ds["x"][j], B) for j in range(d)])
    assert np.array_equal(gb, ob)
    del ds
    n = 1_200_003
    say(f"workload 5: {n} fresh events")
    x = make_apply_chunk(7, n)["x"]
    codes = fb.bin_transform(dev(x), ob)
    xb = np.stack([O.encode(x[j], ob[j]) for j in range(d)]).astype(np.uint8)
    assert np.array_equal(codes.numpy(), xb)
    f = random_forest(T, D, d, B, seed=5)
    model = fb.Model.from_arrays(f["cut_feature"], f["cut_bin"], f["leaf"], f["f0"], d, B)
    score = torch.empty(n, dtype=torch.float64, device="cuda")
    p = fb.apply(model, codes, score=score)
    m = 200_000
    om = O.Model(D, B, d, f["f0"], f["cut_feature"], f["cut_bin"], np.zeros_like(f["leaf"][:, 1:]),
                 f["leaf"])
    say(f"workload 5: oracle apply of the first {m} events")
    op, oF = O.apply(om, xb[:, :m])
    assert np.array_equal(score[:m].cpu().numpy(), oF)
    pg = p[:m].cpu().numpy()
    assert np.max(np.abs(pg.astype(np.float64) - op)) <= 1e-5
    np.testing.assert_array_max_ulp(pg, op, maxulp=1)
    pa = p.cpu().numpy()
    assert np.all((pa > 0.0) & (pa < 1.0))


# ----------------------------------------------------------- float apply
def _edge_events(b, extra, rng):
    """Every boundary, its float32 neighbours above and below, +-0 and +-inf,
    then events drawn from a sample; float32 [d][m]."""
    vals = []
    for j in range(b.shape[0]):
        col = np.concatenate([b[j], np.nextafter(b[j], np.float32(np.inf)),
                              np.nextafter(b[j], np.float32(-np.inf)),
                              np.array([0.0, -0.0, np.inf, -np.inf], np.float32)])
        vals.append(col.astype(np.float32))
    m = max(len(v) for v in vals)
    x = np.stack([np.resize(v, m) for v in vals]).astype(np.float32)
    x = np.concatenate([x, extra[:, rng.integers(0, extra.shape[1], 20_000)]], axis=1)
    return np.ascontiguousarray(x)


@pytest.mark.parametrize("T,D", [(50, 1), (400, 3), (30, 4), (20, 7)])
def test_apply_float_matches_binned_apply_and_oracle(T, D):
    """Section 2.2's inverse transform: fbdt_apply_float on raw values equals
    fbdt_apply on the codes of fbdt_bin_transform bit for bit, and the
    oracle's threshold apply, on values at, just above and just below every
    boundary of a training sample with tied and discrete features."""
    B = 256
    ds = make_training_set(4, n_events=40_001)
    d = ds["x"].shape[0]
    rng = np.random.default_rng(T + D)
    gb, _ = fb.bin(dev(ds["x"]), B)
    x = _edge_events(gb, ds["x"], rng)
    n = x.shape[1]
    say(f"apply_float T={T} D={D} n={n}")
    f = random_forest(T, D, d, B, seed=3 * T + D)
    model = fb.Model.from_arrays(f["cut_feature"], f["cut_bin"], f["leaf"], f["f0"], d, B,
                                 boundaries=gb)
    xs = dev(x)
    sf = torch.empty(n, dtype=torch.float64, device="cuda")
    pf = fb.apply_float(model, xs, score=sf).cpu().numpy()
    codes = fb.bin_transform(xs, gb)
    sb = torch.empty(n, dtype=torch.float64, device="cuda")
    pb = fb.apply(model, codes, score=sb).cpu().numpy()
    assert np.array_equal(sf.cpu().numpy(), sb.cpu().numpy())
    assert np.array_equal(pf, pb)
    om = O.Model(D, B, d, f["f0"], f["cut_feature"], f["cut_bin"], np.zeros_like(f["leaf"][:, 1:]),
                 f["leaf"])
    op, oF = O.apply_thresholds(om, x, gb)
    assert np.array_equal(sf.cpu().numpy(), oF)
    np.testing.assert_array_max_ulp(pf, op, maxulp=1)


def test_apply_float_on_a_fitted_model_with_row_stride():
    """A fitted model gets its training boundaries; fresh events in a padded
    row layout (ldx > n) score as their codes do."""
    spec = CONFIGS[1]
    ds = make_training_set(1)
    bounds, codes = fb.bin(dev(ds["x"]), spec.n_bins)
    model = fb.fit(codes, dev(ds["y"]), spec.n_bins, spec.depth, spec.n_trees, spec.shrinkage,
                   spec.subsample, spec.fit_seed)
    with pytest.raises(fb.FbdtError):
        fb.apply_float(model, dev(ds["x"]))          # no boundaries yet
    model.set_boundaries(bounds)
    d, n = ds["x"].shape
    big = torch.zeros((d, n + 37), dtype=torch.float32, device="cuda")
    big[:, :n] = dev(ds["x"])
    xv = big[:, :n]
    pf = fb.apply_float(model, xv).cpu().numpy()
    pb = fb.apply(model, codes).cpu().numpy()
    assert np.array_equal(pf, pb)
    bad = bounds.copy()
    bad[0, 3] = bad[0, 2] - 1.0
    with pytest.raises(fb.FbdtError):
        model.set_boundaries(bad)


# ------------------------------------------------------------- importance
def test_feature_and_event_importance_match_oracle():
    """Section 4.3: global importance (gains summed per feature) and each
    event's importance (gains on its path) of a fitted model and of a random
    deep forest, against the oracle, exactly (the same float64 sums in the
    same order)."""
    spec = CONFIGS[2]
    ds = make_training_set(2, n_events=60_013)
    B = spec.n_bins
    bounds, codes = fb.bin(dev(ds["x"]), B)
    model = fb.fit(codes, dev(ds["y"]), B, spec.depth, 30, spec.shrinkage, spec.subsample,
                   spec.fit_seed)
    gm = model.export()
    om = _oracle_model(gm)
    assert np.array_equal(fb.feature_importance(model), O.feature_importance(om))
    xb = codes.numpy()
    ei = fb.event_importance(model, codes).cpu().numpy()
    assert np.array_equal(ei, O.event_importance(om, xb))
    rng = np.random.default_rng(11)
    T, D, d, n = 20, 7, 30, 5003
    f = random_forest(T, D, d, B, seed=12)
    gain = rng.exponential(1.0, f["cut_feature"].shape)
    model = fb.Model.from_arrays(f["cut_feature"], f["cut_bin"], f["leaf"], f["f0"], d, B,
                                 gain=gain)
    xr = rng.integers(0, B, (d + 3, n)).astype(np.uint8)     # more rows than features
    codes = fb.Codes.from_numpy(xr)
    ei = fb.event_importance(model, codes).cpu().numpy()
    om = O.Model(D, B, d, f["f0"], f["cut_feature"], f["cut_bin"], gain, f["leaf"])
    assert np.array_equal(ei[:d], O.event_importance(om, xr[:d]))
    assert not ei[d:].any()


# ------------------------------------------------ hand-worked examples
def test_hand_worked_examples_on_the_gpu():
    """The fixtures worked by hand from the paper's definitions, through the
    C ABI: the depth-1 example (binning, the cut, the boost weights and P of
    two trees), its missing-value variant (section 4.2: code 255, the root's
    boost weight for the stopped event), and the exclusive-or table of
    section 4.3 (a zero-gain root cut, gains 0.5 below it, importance)."""
    from tests.golden_io import read_fixture
    _, ex = read_fixture("hand_depth1.txt")
    x = np.array(ex["x"], np.float32)[None, :]
    y = np.array(ex["y"], np.int8)
    bounds, codes = fb.bin(dev(x), 4)
    assert bounds[0].tolist() == ex["boundaries"]
    assert codes.numpy()[0].tolist() == ex["bins"]
    m = fb.fit(codes, dev(y), 4, 1, 2, 1.0, 1.0, 0).export()
    assert int(m["cut_bin"][0, 0]) == int(ex["tree1_cut"][0])
    assert np.allclose(m["leaf"][0], ex["tree1_leaves"], rtol=1e-15)
    assert np.allclose(m["gain"][0, 0], ex["tree1_gains"][0], rtol=1e-15)
    assert int(m["cut_bin"][1, 0]) == int(ex["tree2_cut_eta1"][0])
    assert np.allclose(m["leaf"][1], ex["tree2_leaves_eta1"], atol=1e-6)
    p = fb.apply(fb.fit(codes, dev(y), 4, 1, 2, 1.0, 1.0, 0), codes).cpu().numpy()
    assert np.allclose(p[[0, 2, 4]], ex["tree2_p_eta1"], atol=1e-6)

    _, ex = read_fixture("hand_missing.txt")
    x = np.array(ex["x"], np.float32)[None, :]
    y = np.array(ex["y"], np.int8)
    bounds, codes = fb.bin(dev(x), 4)
    assert bounds[0].tolist() == ex["boundaries"]
    assert codes.numpy()[0].tolist() == [int(v) for v in ex["bins"]]
    model = fb.fit(codes, dev(y), 4, 1, 1, 1.0, 1.0, 0)
    m = model.export()
    assert int(m["cut_bin"][0, 0]) == int(ex["cut"][0])
    assert np.allclose(m["leaf"][0], ex["leaves"], rtol=1e-15)
    assert np.allclose(m["inner"][0], ex["root_value"], atol=1e-15)
    assert np.allclose(fb.apply(model, codes).cpu().numpy(), ex["p"], atol=1e-7)
    model.set_boundaries(bounds)
    assert np.allclose(fb.apply_float(model, dev(x)).cpu().numpy(), ex["p"], atol=1e-7)

    rows, ex = read_fixture("xor_table3.txt")
    t = np.array(rows, np.float32)
    x = np.ascontiguousarray(t[:, :2].T)
    y = np.where(t[:, 2] > 0, 1, -1).astype(np.int8)
    bounds, codes = fb.bin(dev(x), 2)
    model = fb.fit(codes, dev(y), 2, 2, 1, 1.0, 1.0, 0)
    m = model.export()
    assert (int(m["cut_feature"][0, 0]), int(m["cut_bin"][0, 0])) == tuple(
        int(v) for v in ex["root_cut"])
    assert m["gain"][0, 0] == ex["root_gain"][0]
    for k in (1, 2):
        assert (int(m["cut_feature"][0, k]), int(m["cut_bin"][0, k])) == tuple(
            int(v) for v in ex["layer2_cut"])
        assert np.isclose(m["gain"][0, k], ex["layer2_gain"][0], rtol=1e-15)
    p = fb.apply(model, codes).cpu().numpy()
    assert np.allclose(p[y > 0], ex["p_signal"][0], atol=1e-7)
    assert np.allclose(p[y < 0], ex["p_background"][0], atol=1e-7)
    assert np.allclose(fb.feature_importance(model), ex["importance"], rtol=1e-15)
    ei = fb.event_importance(model, codes).cpu().numpy()
    assert np.allclose(ei, np.array(ex["event_importance"])[:, None], rtol=1e-15)


# ------------------------------------------------------------------ errors
def test_errors_are_reported():
    n, d, B = 1000, 3, 16
    rng = np.random.default_rng(0)
    codes = fb.Codes.from_numpy(rng.integers(0, B, (d, n)).astype(np.uint8))
    y = np.where(np.arange(n) % 2 == 0, 1, -1).astype(np.int8)
    bad = y.copy()
    bad[5] = 0
    with pytest.raises(fb.FbdtError) as ei:
        fb.fit(codes, dev(bad), B, 2, 2)
    assert ei.value.status == "FBDT_E_LABEL"
    with pytest.raises(fb.FbdtError) as ei:
        fb.fit(codes, dev(np.ones(n, np.int8)), B, 2, 2)
    assert ei.value.status == "FBDT_E_LABEL"
    w = np.ones(n, np.float32)
    w[y > 0] = -0.5                                    # signal total negative
    w[0] = 1.0
    with pytest.raises(fb.FbdtError) as ei:
        fb.fit(codes, dev(y), B, 2, 2, w=dev(w))
    assert ei.value.status == "FBDT_E_LABEL"
    w = np.ones(n, np.float32)
    w[3] = np.inf
    with pytest.raises(fb.FbdtError) as ei:
        fb.fit(codes, dev(y), B, 2, 2, w=dev(w))
    assert ei.value.status == "FBDT_E_WEIGHT"
    w[3] = np.nan
    with pytest.raises(fb.FbdtError) as ei:
        fb.fit(codes, dev(y), B, 2, 2, w=dev(w))
    assert ei.value.status == "FBDT_E_WEIGHT"
    with pytest.raises(fb.FbdtError) as ei:
        fb.fit(codes, dev(y), 8, 2, 2)                  # codes up to 15 with n_bins = 8
    assert ei.value.status == "FBDT_E_INVAL"
    with pytest.raises(fb.FbdtError) as ei:
        fb.fit(codes, dev(y), B, 8, 2)
    assert ei.value.status == "FBDT_E_INVAL"
    model = fb.fit(codes, dev(y), B, 2, 2)
    small = fb.Codes.from_numpy(np.zeros((2, 10), np.uint8))
    with pytest.raises(fb.FbdtError) as ei:
        fb.apply(model, small)
    assert ei.value.status == "FBDT_E_SHAPE"
    with pytest.raises(fb.FbdtError) as ei:
        fb.Model.from_arrays(np.array([[5]], np.uint8), np.array([[1]], np.uint8),
                             np.zeros((1, 2)), 0.0, 3, 16)
    assert ei.value.status == "FBDT_E_INVAL"


def test_allocation_failure_reports_device_error_and_leaves_the_library_usable():
    """Option fail_alloc makes the library's next device allocations fail as
    an exhausted device would: the fit (its scratch, released by the option
    so that the fit must allocate) and the first apply of a new model (its
    device copy) return FBDT_E_DEVICE, with their outputs untouched; once the
    count is spent the same calls succeed and match the oracle."""
    ds = make_training_set(1)
    spec = CONFIGS[1]
    B, D, T = spec.n_bins, spec.depth, spec.n_trees
    ob, xb = O.bin_features(ds["x"], B)
    codes = fb.Codes.from_numpy(xb)
    y = dev(ds["y"])
    say("allocation failure: fit")
    fb.set_option("fail_alloc", 1)
    try:
        with pytest.raises(fb.FbdtError) as ei:
            fb.fit(codes, y, B, D, T, spec.shrinkage, spec.subsample, spec.fit_seed)
        assert ei.value.status == "FBDT_E_DEVICE"
    finally:
        fb.set_option("fail_alloc", 0)
    model = fb.fit(codes, y, B, D, T, spec.shrinkage, spec.subsample, spec.fit_seed)
    gm = model.export()
    om = O.fit(xb, ds["y"], ds["v"], D, T, spec.shrinkage, spec.subsample, spec.fit_seed, B)
    assert np.array_equal(gm["cut_feature"], om.cut_feature)
    assert np.array_equal(gm["cut_bin"], om.cut_bin)
    say("allocation failure: first apply of a new model")
    fresh = fb.Model.from_arrays(gm["cut_feature"], gm["cut_bin"], gm["leaf"], gm["f0"],
                                 gm["n_features"], B)
    prob = torch.full((codes.n,), -1.0, dtype=torch.float32, device="cuda")
    fb.set_option("fail_alloc", 1)
    try:
        with pytest.raises(fb.FbdtError) as ei:
            fb.apply(fresh, codes, prob=prob)
        assert ei.value.status == "FBDT_E_DEVICE"
    finally:
        fb.set_option("fail_alloc", 0)
    assert bool((prob == -1.0).all())
    p = fb.apply(fresh, codes, prob=prob).cpu().numpy()
    op, _ = O.apply(om, xb)
    assert np.max(np.abs(p.astype(np.float64) - op)) <= 1e-5


def test_apply_float_nan_without_inner_weights_takes_the_left_branch():
    """In a model without inner weights a NaN value fails every threshold
    test x >= b (section 2.2) and goes left at every node that cuts on it:
    fbdt_apply_float equals fbdt_apply on codes where NaN is code 0 (not the
    code 255 of fbdt_bin_transform, which goes right), bit for bit, and the
    oracle's threshold apply."""
    B, D, T, d, n = 64, 3, 50, 6, 5001
    rng = np.random.default_rng(12)
    clean = rng.normal(size=(d, 20_000)).astype(np.float32)
    gb = np.stack([O.quantile_boundaries(clean[j], B) for j in range(d)])
    x = rng.normal(size=(d, n)).astype(np.float32)
    x[rng.random(x.shape) < 0.1] = np.nan
    f = random_forest(T, D, d, B, seed=11)
    model = fb.Model.from_arrays(f["cut_feature"], f["cut_bin"], f["leaf"], f["f0"], d, B,
                                 boundaries=gb)
    say(f"apply_float with NaN, no inner weights: n={n} d={d} T={T}")
    sf = torch.empty(n, dtype=torch.float64, device="cuda")
    pf = fb.apply_float(model, dev(x), score=sf).cpu().numpy()
    codes = np.stack([O.encode(x[j], gb[j]) for j in range(d)])
    assert (codes[np.isnan(x)] == 255).all()
    codes[np.isnan(x)] = 0
    sb = torch.empty(n, dtype=torch.float64, device="cuda")
    pb = fb.apply(model, fb.Codes.from_numpy(codes), score=sb).cpu().numpy()
    assert np.array_equal(pf, pb) and torch.equal(sf, sb)
    om = O.Model(D, B, d, f["f0"], f["cut_feature"], f["cut_bin"],
                 np.zeros_like(f["leaf"][:, 1:]), f["leaf"])
    op, oF = O.apply_thresholds(om, x, gb)
    assert np.array_equal(sf.cpu().numpy(), oF)
    np.testing.assert_array_max_ulp(pf, op, maxulp=1)
