"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these tests compares the oracle with itself: each uses a hand-worked
value, a table of the paper, brute force, a closed form, an invariant, or a
special case that reduces to a library routine (scipy, scikit-learn).
"""
import numpy as np
import pytest
from scipy.special import expit
from scipy.stats import rankdata

from oracle import fbdt_oracle as O
from tests.golden_io import read_fixture


# ---------------------------------------------------------------- SplitMix64
_SM64_1234567 = [6457827717110365317, 3203168211198807973, 9817491932198370423,
                 4593380528125082431, 16408922859458223821]


def test_splitmix64_published_outputs():
    # Reference outputs of SplitMix64 (Steele, Lea & Flood 2014) as published
    # with the reference C implementation: seed 0 and seed 1234567.
    assert int(O.splitmix64(0, [0])[0]) == 0xE220A8397B1DCDAF
    got = [int(z) for z in O.splitmix64(1234567, np.arange(5))]
    assert got == _SM64_1234567


def _u_by_hand(out: int) -> float:
    # the top 53 bits of a published output, as an exact integer times 2^-53
    return float(out >> 11) * 2.0 ** -53


def test_subsample_mask_pins_the_53_bit_mapping_and_counter_layout():
    """The reading of section 1.4: event i of tree t is sampled iff
    u(t N + i) < alpha, with u the top 53 bits of SplitMix64 output number
    t N + i over 2^53.  Derived by hand from the published outputs for seed
    1234567 (outputs 0..4): alpha just above each u samples the event, alpha
    equal to it or just below does not.  Fails for the low 53 bits, for a
    rounding of the top bits, and for an i T + t or i + t counter."""
    u = [_u_by_hand(o) for o in _SM64_1234567]
    assert np.array_equal(O.uniform53(1234567, np.arange(5)), np.array(u))
    seed = 1234567

    def above(x):
        return float(np.nextafter(x, 2.0))

    def below(x):
        return float(np.nextafter(x, -1.0))

    # one event per tree: tree t reads output t
    for t in range(5):
        assert bool(O.subsample_mask(seed, t, 1, above(u[t]))[0])
        assert not bool(O.subsample_mask(seed, t, 1, u[t])[0])
        assert not bool(O.subsample_mask(seed, t, 1, below(u[t]))[0])
    # five events of tree 0: event i reads output i
    for i in range(5):
        m_hi = O.subsample_mask(seed, 0, 5, above(u[i]))
        m_at = O.subsample_mask(seed, 0, 5, u[i])
        assert m_hi.tolist() == [u[k] < above(u[i]) for k in range(5)]
        assert m_at.tolist() == [u[k] < u[i] for k in range(5)]
        assert bool(m_hi[i]) and not bool(m_at[i])
    # tree 1 of two events reads outputs 2 and 3; tree 2 of one event output 2
    for a in sorted(u):
        assert O.subsample_mask(seed, 1, 2, above(a)).tolist() == [u[2] <= a, u[3] <= a]
        assert O.subsample_mask(seed, 2, 1, above(a)).tolist() == [u[2] <= a]
    # the published outputs differ from their low-53-bit images here
    assert any(float(o & ((1 << 53) - 1)) * 2.0 ** -53 != x for o, x in zip(_SM64_1234567, u))


def test_subsample_mask_statistics():
    n, alpha = 200_000, 0.5
    m0 = O.subsample_mask(7, 0, n, alpha)
    m1 = O.subsample_mask(7, 1, n, alpha)
    sd = np.sqrt(n * alpha * (1 - alpha))
    assert abs(m0.sum() - n * alpha) < 5 * sd
    # trees draw independent samples: the overlap is alpha^2
    assert abs((m0 & m1).sum() - n * alpha * alpha) < 5 * np.sqrt(n * 0.25 * 0.75)
    u = O.uniform53(3, np.arange(100_000))
    assert 0.0 <= u.min() and u.max() < 1.0
    assert abs(u.mean() - 0.5) < 5 * np.sqrt(1 / 12 / u.size)
    assert O.subsample_mask(9, 4, 1000, 1.0).all()
    m = O.subsample_mask(9, 4, 100_000, 0.2)
    assert abs(m.mean() - 0.2) < 0.01


# ------------------------------------------------------------------- binning
def _brute_bins(col, n_bins):
    s = sorted(float(v) for v in col)
    n = len(s)
    b = [s[(k * n) // n_bins] for k in range(1, n_bins)]
    return b, [sum(1 for bk in b if bk <= float(v)) for v in col]


@pytest.mark.parametrize("n,n_bins,seed", [(37, 4, 0), (64, 8, 1), (100, 16, 2), (9, 2, 3)])
def test_binning_brute_force(n, n_bins, seed):
    rng = np.random.default_rng(seed)
    col = rng.normal(size=n).astype(np.float32)
    col[: n // 5] = col[n // 5]                         # a block of ties
    b_ref, bins_ref = _brute_bins(col, n_bins)
    b = O.quantile_boundaries(col, n_bins)
    assert np.array_equal(b, np.array(b_ref, np.float32))
    assert O.encode(col, b).tolist() == bins_ref


def test_binning_equal_counts_for_distinct_values():
    # section 2.2 / Fig. 3: equal-frequency bins hold equal counts
    for n, n_bins in [(1000, 16), (1003, 7), (65_537, 256), (500, 256)]:
        col = np.random.default_rng(n).permutation(n).astype(np.float32)
        _, codes = O.bin_features(col[None, :], n_bins)
        counts = np.bincount(codes[0], minlength=n_bins)
        assert set(counts.tolist()) <= {n // n_bins, -(-n // n_bins)}
        assert counts.sum() == n


def test_binning_ties_share_a_bin_and_empty_bins_are_kept():
    col = np.repeat(np.array([0.0, 1.0, 2.0], np.float32), [500, 300, 200])
    b, codes = O.bin_features(col[None, :], 16)
    for value in (0.0, 1.0, 2.0):
        assert len(set(codes[0][col == value].tolist())) == 1
    assert len(set(codes[0].tolist())) == 3
    # values below every boundary go to bin 0, +-inf to the ends
    assert O.encode(np.array([-np.inf, np.inf], np.float32), b[0]).tolist() == [0, 15]
    # NaN (section 4.2) takes the reserved code 255, which needs B <= 255
    assert O.encode(np.array([np.nan], np.float32), b[0]).tolist() == [255]
    b256 = O.quantile_boundaries(np.arange(1000, dtype=np.float32), 256)
    with pytest.raises(ValueError):
        O.encode(np.array([np.nan], np.float32), b256)


def test_binning_monotone_transform_invariance():
    # section 2.2: trees only use the order statistic of the features
    rng = np.random.default_rng(5)
    x = rng.normal(size=(3, 2000)).astype(np.float32)
    x[1, :300] = 0.25
    ranks = np.stack([rankdata(x[j], method="min") for j in range(3)]).astype(np.float32)
    for xt in (x * np.float32(2.0), ranks):
        _, c0 = O.bin_features(x, 32)
        _, c1 = O.bin_features(xt, 32)
        assert np.array_equal(c0, c1)


# --------------------------------------------------------- XOR, Table 3
def test_xor_table3():
    rows, ex = read_fixture("xor_table3.txt")
    rows = np.array(rows)
    x = rows[:, :2].T.astype(np.float32)
    y = np.where(rows[:, 2] > 0, 1, -1).astype(np.int8)
    _, xb = O.bin_features(x, 2)
    assert np.array_equal(xb, x.astype(np.uint8))
    m = O.fit(xb, y, np.ones(4, np.float32), depth=2, n_trees=1, shrinkage=1.0,
              subsample=1.0, seed=0, n_bins=2)
    assert (m.cut_feature[0, 0], m.cut_bin[0, 0]) == tuple(int(v) for v in ex["root_cut"])
    assert m.gain[0, 0] == ex["root_gain"][0]
    for k in (1, 2):
        assert (m.cut_feature[0, k], m.cut_bin[0, k]) == tuple(int(v) for v in ex["layer2_cut"])
        assert m.gain[0, k] == ex["layer2_gain"][0]
    p, _ = O.apply(m, xb)
    sig = y > 0
    assert np.allclose(p[sig], ex["p_signal"][0], rtol=0, atol=1e-7)
    assert np.allclose(p[~sig], ex["p_background"][0], rtol=0, atol=1e-7)
    assert np.allclose(O.feature_importance(m), ex["importance"])
    ei = O.event_importance(m, xb)
    assert np.allclose(ei, np.array(ex["event_importance"])[:, None])


# ------------------------------------------------ hand-worked depth-1 example
def _hand_case():
    _, ex = read_fixture("hand_depth1.txt")
    x = np.array(ex["x"], np.float32)[None, :]
    y = np.array(ex["y"], np.int8)
    return x, y, ex


def test_hand_example_binning_histograms_gains():
    x, y, ex = _hand_case()
    b, xb = O.bin_features(x, 4)
    assert b[0].tolist() == ex["boundaries"]
    assert xb[0].tolist() == ex["bins"]
    w = np.ones(8, np.float32)
    H = O.histogram(xb, np.ones(8, np.int64), w, y > 0, 0, 4)
    assert H[0, 0, :, 0].tolist() == ex["hist_signal"]
    assert H[0, 0, :, 1].tolist() == ex["hist_background"]
    S, Bk = O.cumulative(H)
    assert S[0, 0].tolist() == ex["cph_signal"]
    assert Bk[0, 0].tolist() == ex["cph_background"]
    g = O.split_gains(S, Bk)
    assert np.allclose(g[0, 0], ex["tree1_gains"], rtol=0, atol=1e-15)
    f, c, _ = O.best_cuts(g)
    assert (int(f[0]), int(c[0])) == (0, int(ex["tree1_cut"][0]))


@pytest.mark.parametrize("eta", [1.0, 0.1])
def test_hand_example_two_trees(eta):
    x, y, ex = _hand_case()
    _, xb = O.bin_features(x, 4)
    trace = []
    m = O.fit(xb, y, np.ones(8, np.float32), depth=1, n_trees=2, shrinkage=eta,
              subsample=1.0, seed=0, n_bins=4, trace=trace)
    assert m.f0 == 0.0
    assert int(m.cut_bin[0, 0]) == int(ex["tree1_cut"][0])
    assert np.allclose(m.leaf[0] / eta, ex["tree1_leaves"], rtol=1e-15)
    g2 = O.split_gains(*O.cumulative(trace[1]["H"]))[0, 0]
    if eta == 1.0:
        p1, _ = O.apply(m, xb, n_trees=1)
        assert np.allclose(p1[[0, 7]], ex["tree1_p_eta1"], atol=1e-7)
        assert np.allclose(g2, ex["tree2_gains_eta1"], atol=1e-6)
        assert int(m.cut_bin[1, 0]) == int(ex["tree2_cut_eta1"][0])
        assert np.allclose(m.leaf[1], ex["tree2_leaves_eta1"], atol=1e-6)
        p2, _ = O.apply(m, xb)
        assert np.allclose(p2[[0, 2, 4]], ex["tree2_p_eta1"], atol=1e-6)
    else:
        p1, _ = O.apply(m, xb, n_trees=1)
        assert np.allclose(p1[[0, 7]], ex["tree1_p_eta01"], atol=1e-6)
        assert np.allclose(g2, ex["tree2_gains_eta01"], atol=1e-6)
        assert int(m.cut_bin[1, 0]) == int(ex["tree2_cut_eta01"][0])


def test_hand_missing_value_example():
    """Section 4.2: the hand-worked depth-1 example with one value missing
    (tests/golden/hand_missing.txt): boundaries over the other values, NaN
    code 255 out of the histograms, the same gains, the NaN event stopping at
    the root with the root's boost weight."""
    _, ex = read_fixture("hand_missing.txt")
    x = np.array(ex["x"], np.float32)[None, :]
    y = np.array(ex["y"], np.int8)
    b, xb = O.bin_features(x, 4)
    assert b[0].tolist() == ex["boundaries"]
    assert xb[0].tolist() == [int(v) for v in ex["bins"]]
    H = O.histogram(xb, np.ones(8, np.int64), np.ones(8, np.float32), y > 0, 0, 4)
    assert H[0, 0, :, 0].tolist() == ex["hist_signal"]
    assert H[0, 0, :, 1].tolist() == ex["hist_background"]
    g = O.split_gains(*O.cumulative(H))[0, 0]
    assert np.allclose(g, ex["gains"], rtol=0, atol=1e-15)
    m = O.fit(xb, y, np.ones(8, np.float32), depth=1, n_trees=1, shrinkage=1.0,
              subsample=1.0, seed=0, n_bins=4)
    assert int(m.cut_bin[0, 0]) == int(ex["cut"][0])
    assert np.allclose(m.leaf[0], ex["leaves"], rtol=1e-15)
    assert m.inner is not None and np.allclose(m.inner[0], ex["root_value"], atol=1e-15)
    p, _ = O.apply(m, xb)
    assert np.allclose(p, ex["p"], atol=1e-7)
    pt, _ = O.apply_thresholds(m, x, b)
    assert np.array_equal(pt, p)
    # the missing event's path has no applied cut: no importance
    assert O.event_importance(m, xb)[0].tolist() == [g[1]] * 3 + [0.0] + [g[1]] * 4


def test_missing_values_leave_other_features_and_events_unchanged():
    """Section 4.2: NaN values are ignored.  A feature that is NaN for every
    event never moves an event (all stop at the root when it is cut on), so
    a sample with one extra all-NaN feature placed last, on which the best
    cut never falls when the other features separate, fits the same trees
    as without it; and blanking one value leaves the other features'
    histograms of the root untouched."""
    from synth import make_training_set
    ds = make_training_set(1, n_events=3000)
    _, xb = O.bin_features(ds["x"], 16)
    x2 = np.concatenate([ds["x"], np.full((1, 3000), np.nan, np.float32)])
    _, xb2 = O.bin_features(x2, 16)
    assert (xb2[-1] == 255).all() and np.array_equal(xb2[:-1], xb)
    m1 = O.fit(xb, ds["y"], ds["v"], 3, 3, 0.1, 1.0, 0, 16)
    m2 = O.fit(xb2, ds["y"], ds["v"], 3, 3, 0.1, 1.0, 0, 16)
    assert np.array_equal(m1.cut_feature, m2.cut_feature)
    assert np.array_equal(m1.cut_bin, m2.cut_bin)
    assert np.allclose(m1.leaf, m2.leaf, rtol=1e-12)
    x3 = ds["x"].copy()
    x3[2, 17] = np.nan
    _, xb3 = O.bin_features(x3, 16)
    w = np.ones(3000, np.float32)
    H1 = O.histogram(xb, np.ones(3000, np.int64), w, ds["y"] > 0, 0, 16)
    H3 = O.histogram(xb3, np.ones(3000, np.int64), w, ds["y"] > 0, 0, 16)
    others = [j for j in range(xb.shape[0]) if j != 2]
    assert np.array_equal(H1[:, others], H3[:, others])
    assert H3[0, 2].sum() == H1[0, 2].sum() - 1.0


def test_hand_example_event_importance():
    """Depth 1, two trees at eta = 1: every event passes the root of each tree,
    so its importance is the sum of the two root gains (both on feature 0)."""
    x, y, ex = _hand_case()
    _, xb = O.bin_features(x, 4)
    m = O.fit(xb, y, np.ones(8, np.float32), depth=1, n_trees=2, shrinkage=1.0,
              subsample=1.0, seed=0, n_bins=4)
    g1 = ex["tree1_gains"][int(ex["tree1_cut"][0]) - 1]
    g2 = ex["tree2_gains_eta1"][int(ex["tree2_cut_eta1"][0]) - 1]
    ei = O.event_importance(m, xb)
    assert np.allclose(ei[0], g1 + g2, atol=1e-6)
    assert np.allclose(O.feature_importance(m), [g1 + g2], atol=1e-6)


def test_hand_example_threshold_apply():
    """The depth-1 hand example's first tree (cut c = 1 at eta = 1) applied
    to the raw values: the test is x >= the first boundary, 3."""
    x, y, ex = _hand_case()
    b, xb = O.bin_features(x, 4)
    m = O.fit(xb, y, np.ones(8, np.float32), depth=1, n_trees=1, shrinkage=1.0,
              subsample=1.0, seed=0, n_bins=4)
    p, _ = O.apply_thresholds(m, x, b)
    assert np.allclose(p[:2], ex["tree1_p_eta1"][0], atol=1e-7)
    assert np.allclose(p[2:], ex["tree1_p_eta1"][1], atol=1e-7)


def test_threshold_apply_equals_binned_apply_on_edge_values():
    """Section 2.2's inverse transform: testing x >= b_j,c gives the same leaf
    as testing bin(x) >= c, with bin(x) = searchsorted(b_j, x, 'right') (the
    library routine), for values on, just below and just above every
    boundary, repeated boundaries (tied training values), +-0 and +-inf."""
    from synth import make_training_set, random_forest
    xt = make_training_set(4, n_events=3001)["x"][:10]
    xt[3, :100] = np.inf
    xt[4, :100] = -np.inf
    xt[5, ::2] = -0.0
    B = 32
    b = np.stack([O.quantile_boundaries(xt[j], B) for j in range(10)])
    vals = []
    for j in range(10):
        col = np.concatenate([b[j], np.nextafter(b[j], np.float32(np.inf)),
                              np.nextafter(b[j], np.float32(-np.inf)),
                              np.array([0.0, -0.0, np.inf, -np.inf], np.float32)])
        vals.append(col.astype(np.float32))
    m = max(len(v) for v in vals)
    x = np.stack([np.resize(v, m) for v in vals]).astype(np.float32)
    rng = np.random.default_rng(1)
    x = np.concatenate([x, xt[:, rng.integers(0, xt.shape[1], 500)]], axis=1)
    codes = np.stack([np.searchsorted(b[j], x[j], side="right") for j in range(10)])
    for D in (1, 3, 6):
        f = random_forest(20, D, 10, B, seed=D)
        om = O.Model(D, B, 10, f["f0"], f["cut_feature"], f["cut_bin"],
                     np.zeros_like(f["leaf"][:, 1:]), f["leaf"])
        _, Ft = O.apply_thresholds(om, x, b)
        _, Fb = O.apply(om, codes.astype(np.uint8))
        assert np.array_equal(Ft, Fb)


def test_negative_weights_cancel_a_positive_copy():
    """Section 4.1: events may carry negative weights.  Appending a copy of
    the sample with weight +a and another with weight -a (same features and
    labels) leaves every histogram, gain, boost weight and score unchanged up
    to float64 rounding, with alpha = 1 (no sampling)."""
    from synth import make_training_set
    ds = make_training_set(1, n_events=2000)
    _, xb = O.bin_features(ds["x"], 16)
    n = xb.shape[1]
    rng = np.random.default_rng(2)
    a = rng.uniform(0.5, 2.0, n).astype(np.float32)
    xb3 = np.concatenate([xb, xb, xb], axis=1)
    y3 = np.concatenate([ds["y"]] * 3)
    v3 = np.concatenate([ds["v"], a, -a]).astype(np.float32)
    m1, F1 = O.fit(xb, ds["y"], ds["v"], 3, 4, 0.1, 1.0, 0, 16, final_score=True)
    m3, F3 = O.fit(xb3, y3, v3, 3, 4, 0.1, 1.0, 0, 16, final_score=True)
    assert np.array_equal(m1.cut_feature, m3.cut_feature)
    assert np.array_equal(m1.cut_bin, m3.cut_bin)
    assert np.allclose(m1.leaf, m3.leaf, rtol=1e-9, atol=1e-12)
    assert np.allclose(F3[:n], F1, rtol=1e-9, atol=1e-12)


# ------------------------------------------------------------- histograms
def _brute_hist(xb, node, w, y, layer, n_bins):
    d, n = xb.shape
    H = np.zeros((1 << layer, d, n_bins, 2))
    for i in range(n):
        for j in range(d):
            H[node[i] - (1 << layer), j, xb[j, i], 0 if y[i] > 0 else 1] += float(w[i])
    return H


@pytest.mark.parametrize("layer", [0, 1, 2])
def test_histogram_brute_force_and_totals(layer):
    rng = np.random.default_rng(layer)
    n, d, nb = 300, 3, 8
    xb = rng.integers(0, nb, (d, n)).astype(np.uint8)
    y = np.where(rng.random(n) < 0.4, 1, -1).astype(np.int8)
    w = rng.uniform(0, 2, n).astype(np.float32)
    w[rng.random(n) < 0.5] = 0                          # unsampled events
    node = rng.integers(1 << layer, 2 << layer, n)
    H = O.histogram(xb, node, w, y > 0, layer, nb)
    assert np.allclose(H, _brute_hist(xb, node, w, y, layer, nb), rtol=1e-14, atol=0)
    tot = H.sum(axis=2)                                 # [node][feature][class]
    for k in range(1 << layer):
        for c, sel in ((0, y > 0), (1, y < 0)):
            ref = float(np.sum(w[(node == (1 << layer) + k) & sel].astype(np.float64)))
            assert np.allclose(tot[k, :, c], ref, rtol=1e-13, atol=1e-300)


# ------------------------------------------------------------- best cuts
def _brute_best(xb, w, y, n_bins):
    """Enumerate every (feature, cut) by partitioning the events directly."""
    d, n = xb.shape

    def G(s, b):
        return 0.0 if s + b == 0 else s * b / (s + b)

    ST = sum(float(w[i]) for i in range(n) if y[i] > 0)
    BT = sum(float(w[i]) for i in range(n) if y[i] < 0)
    best = (-np.inf, None)
    gains = {}
    for j in range(d):
        for c in range(1, n_bins):
            sl = sum(float(w[i]) for i in range(n) if y[i] > 0 and xb[j, i] < c)
            bl = sum(float(w[i]) for i in range(n) if y[i] < 0 and xb[j, i] < c)
            sr = sum(float(w[i]) for i in range(n) if y[i] > 0 and xb[j, i] >= c)
            br = sum(float(w[i]) for i in range(n) if y[i] < 0 and xb[j, i] >= c)
            g = G(ST, BT) - G(sl, bl) - G(sr, br)
            gains[(j, c)] = g
            if g > best[0] + 1e-12:
                best = (g, (j, c))
    return best, gains


@pytest.mark.parametrize("seed", range(12))
def test_best_cut_brute_force(seed):
    rng = np.random.default_rng(100 + seed)
    n = int(rng.integers(2, 64))
    d = int(rng.integers(1, 5))
    nb = int(rng.integers(2, 9))
    xb = rng.integers(0, nb, (d, n)).astype(np.uint8)
    y = np.where(rng.random(n) < 0.5, 1, -1).astype(np.int8)
    w = rng.uniform(0.1, 2, n).astype(np.float32)
    (gbest, jc), gains = _brute_best(xb, w, y, nb)
    g = O.split_gains(*O.cumulative(O.histogram(xb, np.ones(n, int), w, y > 0, 0, nb)))
    for (j, c), ref in gains.items():
        assert abs(g[0, j, c - 1] - ref) <= 1e-12 * max(1.0, abs(ref))
    f, c, best = O.best_cuts(g)
    assert abs(best[0] - gbest) <= 1e-12 * max(1.0, abs(gbest))
    # the oracle's choice is the lowest (feature, cut) among the best
    near = sorted(k for k, v in gains.items() if v >= gbest - 1e-12 * max(1.0, abs(gbest)))
    assert (int(f[0]), int(c[0])) == near[0]


def test_weighted_gini_stump_matches_sklearn():
    # the gain is the weighted Gini decrease: a depth-1 scikit-learn tree with
    # the same sample weights picks the same partition
    from sklearn.tree import DecisionTreeClassifier
    for seed in range(5):
        rng = np.random.default_rng(seed)
        n, d, nb = 3000, 5, 32
        xb = rng.integers(0, nb, (d, n)).astype(np.uint8)
        logit = 0.08 * (xb[0].astype(float) - 16) - 0.05 * (xb[3].astype(float) - 16)
        y = np.where(rng.random(n) < expit(logit), 1, -1).astype(np.int8)
        w = rng.uniform(0.05, 3.0, n).astype(np.float32)
        g = O.split_gains(*O.cumulative(O.histogram(xb, np.ones(n, int), w, y > 0, 0, nb)))
        f, c, _ = O.best_cuts(g)
        clf = DecisionTreeClassifier(criterion="gini", max_depth=1, random_state=0)
        clf.fit(xb.T.astype(np.float64), y, sample_weight=w.astype(np.float64))
        assert clf.tree_.feature[0] == f[0]
        thr = clf.tree_.threshold[0]
        col = xb[f[0]]
        assert np.array_equal(col < c[0], col <= thr)


def test_first_tree_matches_sklearn_classifier():
    # first boosting step, F0 = 0, unit weights, no sub-sampling: every weight
    # is 1 and the terminal boost weight is (S - B) / (S + B) = 2 p_signal - 1
    from sklearn.tree import DecisionTreeClassifier
    rng = np.random.default_rng(11)
    n, d, nb, D = 4000, 4, 64, 3
    xb = rng.integers(0, nb, (d, n)).astype(np.uint8)
    logit = 0.05 * (xb[1].astype(float) - 32) + 0.04 * (xb[2].astype(float) - 32) ** 2 / 32
    score = logit + rng.logistic(size=n)
    y = np.where(score > np.median(score), 1, -1).astype(np.int8)   # exactly 50/50: F0 = 0
    m = O.fit(xb, y, np.ones(n, np.float32), depth=D, n_trees=1, shrinkage=1.0,
              subsample=1.0, seed=0, n_bins=nb)
    assert m.f0 == 0.0
    clf = DecisionTreeClassifier(criterion="gini", max_depth=D, random_state=0)
    clf.fit(xb.T.astype(np.float64), y)
    tr = clf.tree_
    # walk both trees together and compare every partition scikit-learn makes
    stack = [(1, 0, np.arange(n))]
    while stack:
        k, s, idx = stack.pop()
        if tr.children_left[s] < 0:
            continue
        f, c = int(m.cut_feature[0, k - 1]), int(m.cut_bin[0, k - 1])
        assert f == tr.feature[s]
        left = xb[f, idx] < c
        assert np.array_equal(left, xb[f, idx] <= tr.threshold[s])
        stack.append((2 * k, tr.children_left[s], idx[left]))
        stack.append((2 * k + 1, tr.children_right[s], idx[~left]))
    _, F = O.apply(m, xb)
    proba = clf.predict_proba(xb.T.astype(np.float64))[:, list(clf.classes_).index(1)]
    assert np.allclose(F, 2 * proba - 1, rtol=0, atol=1e-12)


# ------------------------------------------------------- boosting recursion
def test_pseudo_response_is_scaled_logistic_residual():
    rng = np.random.default_rng(2)
    F = rng.normal(0, 2, 1000)
    y = np.where(rng.random(1000) < 0.5, 1, -1)
    y01 = (y > 0).astype(float)
    assert np.allclose(O.pseudo_response(y, F), 2 * (y01 - expit(2 * F)), rtol=1e-13, atol=1e-15)


def test_boosting_matches_sklearn_gradient_boosting_one_binary_feature():
    # With one binary feature every tree has the same single partition, so
    # the scores of scikit-learn's log-loss gradient boosting (raw score 2F,
    # Newton-step leaves, log-odds prior) must equal 2F of this method
    # (Friedman's two-class LK_TreeBoost) for every tree and weight choice.
    from sklearn.ensemble import GradientBoostingClassifier
    rng = np.random.default_rng(4)
    n, T, eta = 2000, 6, 0.3
    xb = rng.integers(0, 2, (1, n)).astype(np.uint8)
    y = np.where(rng.random(n) < np.where(xb[0] == 1, 0.7, 0.35), 1, -1).astype(np.int8)
    v = rng.uniform(0.2, 2.0, n).astype(np.float32)
    m, Ffit = O.fit(xb, y, v, depth=1, n_trees=T, shrinkage=eta, subsample=1.0, seed=0,
                    n_bins=2, final_score=True)
    gb = GradientBoostingClassifier(loss="log_loss", learning_rate=eta, n_estimators=T,
                                    max_depth=1, subsample=1.0, random_state=0)
    X = xb.T.astype(np.float64)
    gb.fit(X, y, sample_weight=v.astype(np.float64))
    raw = gb.decision_function(X)
    assert np.allclose(2 * Ffit, raw, rtol=1e-9, atol=1e-12)
    p, F = O.apply(m, xb)
    assert np.allclose(p, gb.predict_proba(X)[:, 1], rtol=0, atol=2e-7)
    assert np.allclose(2 * m.f0, np.log(v[y > 0].sum(dtype=np.float64) / v[y < 0].sum(dtype=np.float64)))


def test_first_tree_closed_form_leaves():
    rng = np.random.default_rng(8)
    n, d, nb = 1000, 3, 16
    xb = rng.integers(0, nb, (d, n)).astype(np.uint8)
    y = np.where(np.arange(n) % 2 == 0, 1, -1).astype(np.int8)
    m = O.fit(xb, y, np.ones(n, np.float32), depth=2, n_trees=1, shrinkage=1.0,
              subsample=1.0, seed=0, n_bins=nb)
    node = np.ones(n, int)
    for layer in range(2):
        lo = (1 << layer) - 1
        node = O.route(node, xb, m.cut_feature[0, lo:lo + (1 << layer)],
                       m.cut_bin[0, lo:lo + (1 << layer)], layer)
    for leaf in range(4):
        sel = node == 4 + leaf
        s, b = int(np.sum(y[sel] > 0)), int(np.sum(y[sel] < 0))
        ref = 0.0 if s + b == 0 else (s - b) / (s + b)
        assert abs(m.leaf[0, leaf] - ref) < 1e-15


# ----------------------------------------------------------- invariants
def _fit_small(xb, y, v, seed=3, alpha=0.5, T=5, D=3, nb=16):
    return O.fit(xb, y, v, depth=D, n_trees=T, shrinkage=0.1, subsample=alpha, seed=seed,
                 n_bins=nb, final_score=True)


def _small_problem(seed=1):
    rng = np.random.default_rng(seed)
    n, d, nb = 3000, 4, 16
    xb = rng.integers(0, nb, (d, n)).astype(np.uint8)
    y = np.where(rng.random(n) < expit(0.2 * (xb[0].astype(float) - 8)), 1, -1).astype(np.int8)
    v = rng.uniform(0.5, 1.5, n).astype(np.float32)
    return xb, y, v


def test_label_swap_symmetry():
    xb, y, v = _small_problem()
    m1, F1 = _fit_small(xb, y, v)
    m2, F2 = _fit_small(xb, (-y).astype(np.int8), v)
    assert np.array_equal(m1.cut_feature, m2.cut_feature)
    assert np.array_equal(m1.cut_bin, m2.cut_bin)
    assert np.allclose(F1, -F2, rtol=1e-12, atol=1e-14)
    p1, _ = O.apply(m1, xb)
    p2, _ = O.apply(m2, xb)
    assert np.allclose(p1, 1 - p2, atol=1e-7)


def test_weight_scale_invariance():
    xb, y, v = _small_problem()
    m1, F1 = _fit_small(xb, y, v)
    m2, F2 = _fit_small(xb, y, v * np.float32(4))
    assert np.array_equal(m1.cut_bin, m2.cut_bin)
    assert np.array_equal(m1.cut_feature, m2.cut_feature)
    assert np.array_equal(m1.leaf, m2.leaf)
    assert np.array_equal(F1, F2)


def test_no_subsampling_removes_randomness():
    xb, y, v = _small_problem()
    m1, _ = _fit_small(xb, y, v, seed=1, alpha=1.0)
    m2, _ = _fit_small(xb, y, v, seed=99, alpha=1.0)
    assert np.array_equal(m1.leaf, m2.leaf)
    m3, _ = _fit_small(xb, y, v, seed=1, alpha=0.5)
    m4, _ = _fit_small(xb, y, v, seed=99, alpha=0.5)
    assert not np.array_equal(m3.leaf, m4.leaf)


def test_apply_reproduces_fit_score():
    xb, y, v = _small_problem()
    m, F = _fit_small(xb, y, v, T=8)
    _, Fa = O.apply(m, xb)
    assert np.array_equal(F, Fa)


def test_resume_from_applied_scores_reproduces_later_trees():
    """Resuming the loop at tree t0 with the scores that apply gives for
    trees 0..t0-1 (equal to the loop's own, pinned above) fits the same later
    trees and final score: the sub-sample depends on the tree index only."""
    xb, y, v = _small_problem()
    m, F = _fit_small(xb, y, v, T=8)
    for t0 in (1, 5):
        head = O.Model(m.depth, m.n_bins, m.n_features, m.f0, m.cut_feature[:t0],
                       m.cut_bin[:t0], m.gain[:t0], m.leaf[:t0])
        _, Ft = O.apply(head, xb)
        m2, F2 = O.fit(xb, y, v, m.depth, 8, 0.1, 0.5, 3, m.n_bins, final_score=True,
                       start=(t0, Ft))
        assert np.array_equal(m2.cut_feature[t0:], m.cut_feature[t0:])
        assert np.array_equal(m2.cut_bin[t0:], m.cut_bin[t0:])
        assert np.array_equal(m2.leaf[t0:], m.leaf[t0:])
        assert not m2.leaf[:t0].any()
        assert np.array_equal(F2, F)


def test_near_tie_sets_on_the_xor_table():
    """Table 3 (section 4.3): at the root both features have gain 0, so the
    root's near-tie set holds both cuts; each layer-2 node has one best cut
    (gain 0.5 against 0)."""
    rows, _ = read_fixture("xor_table3.txt")
    rows = np.array(rows)
    xb = rows[:, :2].T.astype(np.uint8)
    y = np.where(rows[:, 2] > 0, 1, -1).astype(np.int8)
    near = []
    O.fit(xb, y, np.ones(4, np.float32), depth=2, n_trees=1, shrinkage=1.0, subsample=1.0,
          seed=0, n_bins=2, near_ties=near)
    assert len(near) == 1
    t, node, cands = near[0]
    assert (t, node) == (0, 1)
    assert sorted((f, c) for f, c, _ in cands) == [(0, 1), (1, 1)]
    assert all(g == 0.0 for _, _, g in cands)


def test_near_tie_sets_leave_out_repeated_partitions():
    """A feature with an empty bin: cut c whose bin c - 1 is empty makes the
    partition of cut c - 1 and is not a separate candidate."""
    xb = np.array([[0, 0, 2, 2, 3, 3]], np.uint8)      # bin 1 empty: cuts 1 and 2 alike
    y = np.array([-1, -1, 1, 1, 1, -1], np.int8)
    near = []
    m = O.fit(xb, y, np.ones(6, np.float32), depth=1, n_trees=1, shrinkage=1.0, subsample=1.0,
              seed=0, n_bins=4, near_ties=near)
    assert (int(m.cut_feature[0, 0]), int(m.cut_bin[0, 0])) == (0, 1)
    assert near == []


def test_model_invariant_under_monotone_feature_transform():
    rng = np.random.default_rng(6)
    x = rng.normal(size=(3, 2000)).astype(np.float32)
    y = np.where(rng.random(2000) < expit(x[0] - 0.5 * x[2]), 1, -1).astype(np.int8)
    v = np.ones(2000, np.float32)
    _, xb1 = O.bin_features(x, 16)
    ranks = np.stack([rankdata(x[j], method="min") for j in range(3)]).astype(np.float32)
    m1 = O.fit(xb1, y, v, 3, 4, 0.1, 0.5, 0, 16)
    for xt in (x * np.float32(2.0), ranks):
        _, xb2 = O.bin_features(xt, 16)
        m2 = O.fit(xb2, y, v, 3, 4, 0.1, 0.5, 0, 16)
        assert np.array_equal(m1.cut_bin, m2.cut_bin) and np.array_equal(m1.leaf, m2.leaf)


def test_empty_node_takes_first_cut_and_zero_leaves():
    # all events share one bin of every feature: no cut separates anything,
    # every gain is 0, so every node takes (feature 0, cut 1); the side that
    # receives no event gets boost weight 0
    n = 50
    xb = np.full((2, n), 3, np.uint8)
    y = np.where(np.arange(n) % 3 == 0, 1, -1).astype(np.int8)
    m = O.fit(xb, y, np.ones(n, np.float32), depth=2, n_trees=1, shrinkage=1.0,
              subsample=1.0, seed=0, n_bins=8)
    assert m.cut_feature[0].tolist() == [0, 0, 0]
    assert m.cut_bin[0].tolist() == [1, 1, 1]
    assert np.all(m.gain[0] == 0.0)
    assert m.leaf[0, 0] == 0.0 and m.leaf[0, 1] == 0.0 and m.leaf[0, 2] == 0.0
    assert m.leaf[0, 3] != 0.0


def test_apply_hand_built_forest():
    # a depth-2 tree written by hand, traced as in Fig. 1 (left = bin < cut)
    m = O.Model(depth=2, n_bins=8, n_features=2, f0=0.25,
                cut_feature=np.array([[0, 1, 0]], np.uint8),
                cut_bin=np.array([[3, 5, 2]], np.uint8),
                gain=np.zeros((1, 3)),
                leaf=np.array([[0.1, 0.2, 0.3, 0.4]]))
    xb = np.array([[0, 2, 3, 7, 1], [4, 5, 0, 7, 6]], np.uint8)
    # event 0: f0=0<3 -> node 2: f1=4<5 -> leaf 4 (0.1)
    # event 1: f0=2<3 -> node 2: f1=5>=5 -> leaf 5 (0.2)
    # event 2: f0=3>=3 -> node 3: f0=3>=2 -> leaf 7 (0.4)
    # event 3: f0=7>=3 -> node 3: f0=7>=2 -> leaf 7 (0.4)
    # event 4: f0=1<3 -> node 2: f1=6>=5 -> leaf 5 (0.2)
    p, F = O.apply(m, xb)
    ref = 0.25 + np.array([0.1, 0.2, 0.4, 0.4, 0.2])
    assert np.allclose(F, ref, rtol=0, atol=1e-15)
    assert np.allclose(p, expit(2 * ref), rtol=0, atol=1e-7)

