"""CPU oracle for FastBDT's fit and apply path (Keck, arXiv:1609.06119).

TEST INFRASTRUCTURE ONLY.  This module is the slow, plain reference that
the GPU library is checked against.  Only the test suite, the smoke check
and the benchmark's CPU-baseline leg may import it; the library never does
and shares no code with it.

Everything is plain numpy in float64, single-threaded, one step of the
method at a time, in the order the paper describes it:

  binning (section 2.2) -> initial score (section 1.2/1.3, Friedman's
  two-class LK_TreeBoost) -> per tree: sub-sample (section 1.4),
  gradient re-weighting (section 1.3), for each layer: signal/background
  histograms of all nodes and features (sections 1.1 and 2.1), cumulative
  probability histograms, separation gain, best cut, routing (section 1.1,
  Fig. 1) -> terminal boost weights and score update (section 1.3) ->
  apply: traverse, sum, sigmoid (Fig. 1, section 1.3), on bin codes or on
  raw values with the inverse transform of section 2.2.

Where the paper is silent the reading is stated at the function.  Pins:
every function is checked by ``tests/test_oracle_*.py`` against something
other than itself (hand-worked examples, the XOR table of section 4.3,
brute force, closed forms, scikit-learn/scipy special cases and published
SplitMix64 outputs).

Notation: N events, d features, B bins, D depth, T trees, eta shrinkage,
alpha sub-sampling rate.  Node ids are heap-ordered: the root is 1, layer
l (0-based) holds nodes [2^l, 2^(l+1)), leaves are [2^D, 2^(D+1)).
"""
from __future__ import annotations

import dataclasses
import time

import numpy as np

_U64 = np.uint64
_GAMMA = _U64(0x9E3779B97F4A7C15)
_MIX1 = _U64(0xBF58476D1CE4E5B9)
_MIX2 = _U64(0x94D049BB133111EB)


# --------------------------------------------------------------------------
# Random sub-sample (section 1.4).  The paper draws a random fraction alpha
# without replacement per tree but names no generator.  Reading: one
# counter-based Bernoulli draw per (tree, event) from SplitMix64 (Steele,
# Lea & Flood, "Fast splittable pseudorandom number generators", OOPSLA
# 2014); the k-th output (k = 0, 1, ...) of a generator seeded with s is the
# mix of state s + (k + 1) * gamma.
# --------------------------------------------------------------------------
def splitmix64(seed: int, counters) -> np.ndarray:
    """Outputs number ``counters`` (0-based) of SplitMix64 seeded with ``seed``."""
    k = np.asarray(counters, dtype=_U64)
    with np.errstate(over="ignore"):
        z = _U64(seed & 0xFFFFFFFFFFFFFFFF) + (k + _U64(1)) * _GAMMA
        z = (z ^ (z >> _U64(30))) * _MIX1
        z = (z ^ (z >> _U64(27))) * _MIX2
        z = z ^ (z >> _U64(31))
    return z


def uniform53(seed: int, counters) -> np.ndarray:
    """Top 53 bits of each output, scaled to [0, 1)."""
    return (splitmix64(seed, counters) >> _U64(11)).astype(np.float64) * (2.0 ** -53)


def subsample_mask(seed: int, tree: int, n_events: int, alpha: float) -> np.ndarray:
    """Event i is in tree t's sub-sample iff u(t*N + i) < alpha.

    Each event is drawn at most once (no replacement); the sample size is
    Binomial(N, alpha).  alpha = 1 keeps every event.
    """
    k = np.uint64(tree) * np.uint64(n_events) + np.arange(n_events, dtype=_U64)
    return uniform53(seed, k) < alpha


# --------------------------------------------------------------------------
# Equal-frequency binning (section 2.2, Fig. 3).
# Reading: with s the ascending sort of one feature over all N training
# events, boundary k (k = 1..B-1) is s[floor(k*N/B)], and a value x goes to
# bin #{k : b_k <= x}.  Distinct values then fill every bin with floor(N/B)
# or ceil(N/B) events; tied values share a bin; repeated boundaries leave
# empty bins, which are kept.  Comparisons are float32, as stored.
# --------------------------------------------------------------------------
# Missing values (section 4.2).  NaN marks a value that must not inform the
# fit.  Reading: NaN takes the reserved code 255 (so B <= 255 bins when the
# data hold NaN); the boundaries are the order statistics of the feature's
# other values; a NaN never enters the feature's histograms; an event whose
# value of a node's cut feature is NaN stops at that node, which acts as its
# terminal node (its boost weight, computed like a leaf's over the sampled
# events that reached it, is added to F); apply does the same.
MISSING = 255


def missing_allowed(n_bins: int) -> bool:
    return n_bins <= MISSING


def quantile_boundaries(column, n_bins: int) -> np.ndarray:
    """b_k = the value of rank floor(k m / B) among the m non-NaN values of
    the feature (k = 1 .. B - 1); +inf when every value is NaN.  NaN is an
    error unless B <= 255 (section 4.2)."""
    col = np.asarray(column, dtype=np.float32)
    nan = np.isnan(col)
    if nan.any() and not missing_allowed(n_bins):
        raise ValueError("NaN feature values need n_bins <= 255")
    s = np.sort(col[~nan])
    m = s.shape[0]
    if m == 0:
        return np.full(n_bins - 1, np.inf, np.float32)
    k = np.arange(1, n_bins, dtype=np.int64)
    return s[(k * m) // n_bins].astype(np.float32)


def encode(column, boundaries) -> np.ndarray:
    """Bin code of every value: the number of boundaries at or below it;
    NaN takes the reserved code 255 (B <= 255, section 4.2)."""
    col = np.asarray(column, dtype=np.float32)
    b = np.asarray(boundaries, dtype=np.float32)
    nan = np.isnan(col)
    if nan.any() and not missing_allowed(b.shape[0] + 1):
        raise ValueError("NaN feature values need n_bins <= 255")
    code = np.searchsorted(b, col, side="right")
    return np.where(nan, MISSING, code).astype(np.uint8)


def bin_features(x, n_bins: int):
    """Boundaries float32 [d][B-1] and codes uint8 [d][N] of a feature-major sample."""
    x = np.asarray(x, dtype=np.float32)
    bounds = np.stack([quantile_boundaries(x[j], n_bins) for j in range(x.shape[0])])
    codes = np.stack([encode(x[j], bounds[j]) for j in range(x.shape[0])])
    return bounds, codes


# --------------------------------------------------------------------------
# Boosting (sections 1.2-1.3; the paper defers the derivation to Friedman,
# "Greedy function approximation", 2001, two-class LK_TreeBoost).
# Reading: F is half the log-odds; the initial score is
# F0 = 1/2 ln(sum of signal weight / sum of background weight); the
# pseudo-response is y~ = 2y / (1 + exp(2 y F)); a terminal node's boost
# weight is the one-step Newton value sum(v y~) / sum(v |y~| (2 - |y~|));
# P(signal) = 1 / (1 + exp(-2F)).
# --------------------------------------------------------------------------
def initial_score(y, v) -> float:
    y = np.asarray(y)
    v = np.asarray(v, dtype=np.float64)
    s = float(np.sum(v[y > 0]))
    b = float(np.sum(v[y < 0]))
    if not (s > 0.0 and b > 0.0):
        raise ValueError("both classes need positive total weight")
    return 0.5 * np.log(s / b)


def pseudo_response(y, F) -> np.ndarray:
    """y~ = 2y / (1 + exp(2yF)), the negative gradient of the binomial deviance."""
    yf = np.asarray(y, dtype=np.float64)
    return 2.0 * yf / (1.0 + np.exp(2.0 * yf * np.asarray(F, dtype=np.float64)))


def histogram_weights(y, v, ytilde, mask) -> np.ndarray:
    """Re-weighted sample (section 1.3): w_i = fl32(v_i |y~_i|) if sampled, else 0.

    Reading: the boosting step re-weights the original sample, and the tree
    then separates signal from background with these weights.  The weight
    is rounded to float32 once, as stored.
    """
    w = (np.asarray(v, dtype=np.float64) * np.abs(ytilde)).astype(np.float32)
    return np.where(mask, w, np.float32(0.0))


def histogram(xb, node, w, is_signal, layer: int, n_bins: int) -> np.ndarray:
    """Signal and background histograms of every node and feature of one layer.

    H[n][j][k][c] = sum of w over events in node 2^layer + n with bin k in
    feature j and class c (c = 0 signal, c = 1 background); sections 1.1
    and 2.1: one pass over the sample fills all nodes and features of the
    layer.  Sums are float64, in event order.
    """
    xb = np.asarray(xb)
    d = xb.shape[0]
    n_nodes = 1 << layer
    local = np.asarray(node, dtype=np.int64) - n_nodes
    cls = np.where(is_signal, 0, 1)
    w64 = np.asarray(w, dtype=np.float32).astype(np.float64)
    H = np.zeros((n_nodes, d, n_bins, 2))
    # events that stopped at an earlier layer (missing values) are not in
    # the layer; a missing value of feature j is not in feature j's histogram
    here = local >= 0
    for j in range(d):
        code = xb[j].astype(np.int64)
        keep = here & (code < n_bins) if missing_allowed(n_bins) else here
        idx = ((local * n_bins + code) * 2 + cls)[keep]
        H[:, j] = np.bincount(idx, weights=w64[keep], minlength=n_nodes * n_bins * 2).reshape(
            n_nodes, n_bins, 2)
    return H


def cumulative(H):
    """Cumulative probability histograms (section 1.1).

    S[n][j][c] and Bk[n][j][c], c = 0..B: summed signal and background
    weight of the bins below c.  S[..., B] is the node's total.
    """
    n_nodes, d, n_bins, _ = H.shape
    S = np.zeros((n_nodes, d, n_bins + 1))
    Bk = np.zeros((n_nodes, d, n_bins + 1))
    S[:, :, 1:] = np.cumsum(H[:, :, :, 0], axis=2)
    Bk[:, :, 1:] = np.cumsum(H[:, :, :, 1], axis=2)
    return S, Bk


def gini(s, b):
    """G(s, b) = s b / (s + b), zero for an empty side.

    Reading: the paper asks for a separation gain without giving it; this is
    the weighted Gini impurity (s + b) p (1 - p) with p = s / (s + b).
    """
    s = np.asarray(s, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    tot = s + b
    with np.errstate(invalid="ignore", divide="ignore"):
        g = (s * b) / tot
    return np.where(tot == 0.0, 0.0, g)


def split_gains(S, Bk) -> np.ndarray:
    """Separation gain of every candidate cut c = 1..B-1 (section 1.1).

    gain = (G(S_T, B_T) - G(S(c), B(c))) - G(S_T - S(c), B_T - B(c)),
    evaluated in that order; column c - 1 of the result is cut c.  A cut c
    sends bins < c to the left child 2n and bins >= c to the right child
    2n + 1 (Fig. 1: the "x < 3" branch is the left one).
    """
    n_bins = S.shape[2] - 1
    ST = S[:, :, n_bins:n_bins + 1]
    BT = Bk[:, :, n_bins:n_bins + 1]
    Sc = S[:, :, 1:n_bins]
    Bc = Bk[:, :, 1:n_bins]
    return (gini(ST, BT) - gini(Sc, Bc)) - gini(ST - Sc, BT - Bc)


def best_cuts(gains):
    """Per node: the (feature, cut) of highest gain; ties go to the lowest
    feature, then the lowest cut.  Every node is split, even at gain 0 (the
    XOR example of section 4.3 takes a zero-gain cut)."""
    n_nodes, d, nc = gains.shape
    flat = gains.reshape(n_nodes, d * nc)
    arg = np.argmax(flat, axis=1)                 # first maximum = lowest (j, c)
    feat = (arg // nc).astype(np.uint8)
    cut = (arg % nc + 1).astype(np.uint8)
    return feat, cut, flat[np.arange(n_nodes), arg]


def route(node, xb, feat_of_node, cut_of_node, layer: int, missing: bool = False) -> np.ndarray:
    """Send every event to a child: node <- 2 node + [bin(f*) >= c*] (section 1.1).
    With ``missing`` (section 4.2) an event whose code of the cut feature is
    the missing code stays at its node, and an event that stopped at an
    earlier layer stays where it is."""
    node = np.asarray(node, dtype=np.int64)
    local = node - (1 << layer)
    here = local >= 0
    lc = np.where(here, local, 0)
    f = np.asarray(feat_of_node, dtype=np.int64)[lc]
    c = np.asarray(cut_of_node, dtype=np.int64)[lc]
    code = np.asarray(xb)[f, np.arange(node.shape[0])].astype(np.int64)
    child = 2 * node + (code >= c).astype(np.int64)
    if not missing:
        return child
    return np.where(here & (code != MISSING), child, node)


def leaf_values(leaf_local, ytilde, v, mask, n_leaves: int) -> np.ndarray:
    """Terminal boost weights gamma_j = sum(v y~) / sum(v |y~| (2 - |y~|)) over
    the sampled events of leaf j, 0 where the denominator is 0 (section 1.3)."""
    yt = np.asarray(ytilde, dtype=np.float64)
    v64 = np.asarray(v, dtype=np.float64)
    m = np.asarray(mask, dtype=bool)
    idx = np.asarray(leaf_local, dtype=np.int64)[m]
    num = np.bincount(idx, weights=(v64 * yt)[m], minlength=n_leaves)
    a = np.abs(yt)
    den = np.bincount(idx, weights=(v64 * a * (2.0 - a))[m], minlength=n_leaves)
    with np.errstate(invalid="ignore", divide="ignore"):
        g = num / den
    return np.where(den == 0.0, 0.0, g)


def node_values(terminal, ytilde, v, mask, depth: int) -> np.ndarray:
    """Boost weights of every node (section 4.2 reading): for node k the
    Newton step sum(v y~) / sum(v |y~| (2 - |y~|)) over the sampled events
    that reached k (those whose terminal node is k or below it), 0 where the
    denominator is 0.  terminal: heap id of each event's terminal node.
    Returns float64 [2^(D+1) - 1], node k at index k - 1."""
    n_nodes = (2 << depth) - 1
    yt = np.asarray(ytilde, dtype=np.float64)
    v64 = np.asarray(v, dtype=np.float64)
    m = np.asarray(mask, dtype=bool)
    idx = np.asarray(terminal, dtype=np.int64)[m] - 1
    num = np.bincount(idx, weights=(v64 * yt)[m], minlength=n_nodes)
    a = np.abs(yt)
    den = np.bincount(idx, weights=(v64 * a * (2.0 - a))[m], minlength=n_nodes)
    for k in range((1 << depth) - 1, 0, -1):   # inner nodes, bottom up
        num[k - 1] += num[2 * k - 1] + num[2 * k]
        den[k - 1] += den[2 * k - 1] + den[2 * k]
    with np.errstate(invalid="ignore", divide="ignore"):
        g = num / den
    return np.where(den == 0.0, 0.0, g)


@dataclasses.dataclass
class Model:
    """A fitted forest in heap order: node k of tree t at index [t, k - 1]."""

    depth: int
    n_bins: int
    n_features: int
    f0: float
    cut_feature: np.ndarray     # uint8 [T][2^D - 1]
    cut_bin: np.ndarray         # uint8 [T][2^D - 1]
    gain: np.ndarray            # float64 [T][2^D - 1]
    leaf: np.ndarray            # float64 [T][2^D], already multiplied by eta
    inner: np.ndarray | None = None   # float64 [T][2^D - 1] times eta: the boost
                                      # weights of inner nodes, for missing values

    @property
    def n_trees(self) -> int:
        return int(self.leaf.shape[0])


@dataclasses.dataclass
class TieLog:
    """Nodes where a reference cut was adopted because it is a near-tie."""

    adopted: list = dataclasses.field(default_factory=list)
    rejected: list = dataclasses.field(default_factory=list)


def is_near_tie(best_gain: float, other_gain: float, parent_gini: float,
                rtol: float = 1e-6, noise: float = 1e-12) -> bool:
    """True when ``other_gain`` is within ``rtol`` (relative) of the best.

    Gains that are zero mathematically come out as rounding noise of order
    1e-16 times the parent's G, so an absolute floor of ``noise`` times the
    parent's G is added to the relative test.
    """
    return best_gain - other_gain <= rtol * abs(best_gain) + noise * abs(parent_gini)


def _near_tie_candidates(H, g, best, parent, k):
    """Every (feature, cut, gain) of node k that ``is_near_tie`` admits beside
    the best, leaving out cuts c >= 2 whose bin c - 1 is empty in the node
    (they make the same partition as cut c - 1, whose gain they share)."""
    nc = g.shape[2]
    # bin c - 1 of cut c (column c - 1 of g) empty in both classes
    empty = (H[k, :, :nc, 0] == 0.0) & (H[k, :, :nc, 1] == 0.0)
    empty[:, 0] = False                       # cut 1 is never a repeat
    near = is_near_tie(float(best[k]), g[k], float(parent[k])) & ~empty
    return [(int(j), int(c0) + 1, float(g[k, j, c0])) for j, c0 in zip(*np.nonzero(near))]


class _Clock:
    """Wall-clock seconds per named step, summed into a dict (or nothing)."""

    def __init__(self, into: dict | None):
        self.into = into
        self.t = 0.0

    def start(self):
        if self.into is not None:
            self.t = time.perf_counter()

    def stop(self, name: str):
        if self.into is not None:
            now = time.perf_counter()
            self.into[name] = self.into.get(name, 0.0) + (now - self.t)
            self.t = now


def fit(xb, y, v, depth: int, n_trees: int, shrinkage: float, subsample: float,
        seed: int, n_bins: int, reference: Model | None = None, tie_log: TieLog | None = None,
        trace: list | None = None, final_score: bool = False, start=None,
        near_ties: list | None = None, timings: dict | None = None):
    """Stochastic gradient-boosted trees on binned features (sections 1.1-1.4, 2.1).

    ``reference`` (optional) holds another implementation's cuts.  Where that
    cut differs from this function's choice but its gain, computed here, is a
    near tie (``is_near_tie``), this function adopts it and records the node
    in ``tie_log`` so that a layer-by-layer comparison can continue past
    genuine ties; any other difference is recorded as rejected and this
    function keeps its own cut.  ``trace`` (optional list) receives one dict
    per layer with the histogram and chosen cuts.
    ``start`` (optional) = (t0, F): resume the boosting loop at tree t0 with
    the scores F that trees 0..t0-1 left (e.g. ``apply`` of those trees on
    the same events, which reproduces the loop's F exactly); the model's rows
    of the trees before t0 stay zero.  ``near_ties`` (optional list) receives,
    for every node whose near-tie set holds more than its best cut, a tuple
    (tree, heap node, [(feature, cut, gain), ...]) of that set.
    ``timings`` (optional dict) accumulates wall seconds per step: "reweight"
    (sub-sample, pseudo-response, weights), "histogram_l<layer>",
    "scan_l<layer>" (cumulative sums, gains, best cut), "route_l<layer>" and
    "leaf" (boost weights and score update).
    Returns the Model, and the final score F when ``final_score``.
    """
    xb = np.asarray(xb)
    d, n = xb.shape
    y = np.asarray(y)
    v = np.asarray(v, dtype=np.float32)
    is_signal = y > 0
    n_inner = (1 << depth) - 1
    f0 = initial_score(y, v)
    F = np.full(n, f0)
    t_first = 0
    if start is not None:
        t_first, F = int(start[0]), np.array(start[1], dtype=np.float64)
    cut_feature = np.zeros((n_trees, n_inner), np.uint8)
    cut_bin = np.zeros((n_trees, n_inner), np.uint8)
    gain_out = np.zeros((n_trees, n_inner))
    leaf_out = np.zeros((n_trees, 1 << depth))
    # missing values (section 4.2): NaN codes in data binned with B <= 255
    missing = missing_allowed(n_bins) and bool((xb == MISSING).any())
    inner_out = np.zeros((n_trees, (1 << depth) - 1)) if missing else None
    clock = _Clock(timings)
    for t in range(t_first, n_trees):
        clock.start()
        mask = subsample_mask(seed, t, n, subsample)
        yt = pseudo_response(y, F)
        w = histogram_weights(y, v, yt, mask)
        node = np.ones(n, dtype=np.int64)
        clock.stop("reweight")
        for layer in range(depth):
            H = histogram(xb, node, w, is_signal, layer, n_bins)
            clock.stop(f"histogram_l{layer}")
            S, Bk = cumulative(H)
            g = split_gains(S, Bk)
            feat, cut, best = best_cuts(g)
            clock.stop(f"scan_l{layer}")
            lo = (1 << layer) - 1
            if near_ties is not None:
                parent = gini(S[:, 0, n_bins], Bk[:, 0, n_bins])
                for k in range(1 << layer):
                    cands = _near_tie_candidates(H, g, best, parent, k)
                    if len(cands) > 1:
                        near_ties.append((t, (1 << layer) + k, cands))
            if reference is not None:
                parent = gini(S[:, 0, n_bins], Bk[:, 0, n_bins])
                for k in range(1 << layer):
                    rf = int(reference.cut_feature[t, lo + k])
                    rc = int(reference.cut_bin[t, lo + k])
                    if (rf, rc) == (int(feat[k]), int(cut[k])):
                        continue
                    ok = 0 <= rf < d and 1 <= rc < n_bins
                    other = float(g[k, rf, rc - 1]) if ok else -np.inf
                    rec = (t, layer, (1 << layer) + k, (int(feat[k]), int(cut[k]), float(best[k])),
                           (rf, rc, other))
                    if ok and is_near_tie(float(best[k]), other, float(parent[k])):
                        feat[k], cut[k], best[k] = rf, rc, other
                        if tie_log is not None:
                            tie_log.adopted.append(rec)
                    elif tie_log is not None:
                        tie_log.rejected.append(rec)
            cut_feature[t, lo:lo + (1 << layer)] = feat
            cut_bin[t, lo:lo + (1 << layer)] = cut
            gain_out[t, lo:lo + (1 << layer)] = best
            if trace is not None:
                trace.append({"tree": t, "layer": layer, "H": H, "node": node.copy(),
                              "w": w, "feat": feat.copy(), "cut": cut.copy()})
            clock.start()
            node = route(node, xb, feat, cut, layer, missing)
            clock.stop(f"route_l{layer}")
        leaf_local = node - (1 << depth)
        if missing:
            values = shrinkage * node_values(node, yt, v, mask, depth)
            inner_out[t] = values[:(1 << depth) - 1]
            leaf_out[t] = values[(1 << depth) - 1:]
            F = F + values[node - 1]
        else:
            gamma = leaf_values(leaf_local, yt, v, mask, 1 << depth)
            leaf_out[t] = shrinkage * gamma
            F = F + leaf_out[t][leaf_local]
        clock.stop("leaf")
    model = Model(depth, n_bins, d, f0, cut_feature, cut_bin, gain_out, leaf_out, inner_out)
    return (model, F) if final_score else model


def apply(model: Model, xb, n_trees: int | None = None):
    """Score events (Fig. 1; section 1.3): F = F0 + sum over trees of the leaf
    reached, summed in tree order in float64; P(signal) = 1/(1 + exp(-2F)),
    rounded to float32.  Returns (P float32 [N], F float64 [N])."""
    xb = np.asarray(xb)
    n = xb.shape[1]
    T = model.n_trees if n_trees is None else n_trees
    F = np.full(n, model.f0)
    rows = np.arange(n)
    for t in range(T):
        node = np.ones(n, dtype=np.int64)
        done = np.zeros(n, dtype=bool)   # stopped at an inner node (missing value)
        for _ in range(model.depth):
            f = model.cut_feature[t][node - 1].astype(np.int64)
            c = model.cut_bin[t][node - 1].astype(np.int64)
            code = xb[f, rows].astype(np.int64)
            if model.inner is not None:
                done |= code == MISSING
            node = np.where(done, node, 2 * node + (code >= c))
        F = F + _node_value(model, t, node)
    p = (1.0 / (1.0 + np.exp(-2.0 * F))).astype(np.float32)
    return p, F


def _node_value(model: Model, t: int, node):
    """Boost weight (times eta) of heap node ``node`` of tree t: a leaf's, or
    with missing values an inner node's."""
    nleaf = 1 << model.depth
    if model.inner is None:
        return model.leaf[t][node - nleaf]
    allv = np.concatenate([model.inner[t], model.leaf[t]])
    return allv[node - 1]


def apply_thresholds(model: Model, x, boundaries, n_trees: int | None = None):
    """Score float32 events without binning them (section 2.2, the inverse
    of the bin transform): a value's bin is the number of boundaries at or
    below it, so the cut "bin >= c" of feature j is the test x >= b_j,c, the
    c-th smallest training boundary of feature j (boundaries[j][c - 1]).
    Leaf values summed in tree order in float64, as in ``apply``.
    Returns (P float32 [N], F float64 [N])."""
    x = np.asarray(x, dtype=np.float32)
    b = np.asarray(boundaries, dtype=np.float32)
    n = x.shape[1]
    T = model.n_trees if n_trees is None else n_trees
    F = np.full(n, model.f0)
    rows = np.arange(n)
    for t in range(T):
        node = np.ones(n, dtype=np.int64)
        done = np.zeros(n, dtype=bool)   # stopped at an inner node (NaN value)
        for _ in range(model.depth):
            f = model.cut_feature[t][node - 1].astype(np.int64)
            c = model.cut_bin[t][node - 1].astype(np.int64)
            xv = x[f, rows]
            if model.inner is not None:
                done |= np.isnan(xv)
            node = np.where(done, node, 2 * node + (xv >= b[f, c - 1]))
        F = F + _node_value(model, t, node)
    p = (1.0 / (1.0 + np.exp(-2.0 * F))).astype(np.float32)
    return p, F


def feature_importance(model: Model) -> np.ndarray:
    """Global importance: summed separation gain per feature (section 4.3)."""
    imp = np.zeros(model.n_features)
    np.add.at(imp, model.cut_feature.ravel().astype(np.int64), model.gain.ravel())
    return imp


def event_importance(model: Model, xb, n_trees: int | None = None) -> np.ndarray:
    """Importance of every feature for every event (section 4.3): the
    separation gains of the nodes on the event's path through the trees,
    summed per feature of the node's cut, tree by tree in float64.
    Returns float64 [d][N]."""
    xb = np.asarray(xb)
    n = xb.shape[1]
    T = model.n_trees if n_trees is None else n_trees
    imp = np.zeros((model.n_features, n))
    rows = np.arange(n)
    for t in range(T):
        node = np.ones(n, dtype=np.int64)
        done = np.zeros(n, dtype=bool)   # stopped at an inner node (missing value)
        for _ in range(model.depth):
            f = model.cut_feature[t][node - 1].astype(np.int64)
            c = model.cut_bin[t][node - 1].astype(np.int64)
            code = xb[f, rows].astype(np.int64)
            if model.inner is not None:
                done |= code == MISSING
            # a node adds its gain to the events its cut applies to
            imp[f, rows] += np.where(done, 0.0, model.gain[t][node - 1])
            node = np.where(done, node, 2 * node + (code >= c))
    return imp
