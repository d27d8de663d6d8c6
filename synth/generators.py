"""Synthetic stand-ins for the paper's Monte Carlo training sample.

The paper times its fits on a simulated D0 -> K pi pi0 sample (1 M points,
35 features; section 3) and states that the data's nature does not affect
the runtime.  That sample is not available, so five seeded synthetic
workloads stand in for it.  Each generator returns float32 features stored
feature-major (``x[j, i]`` is feature ``j`` of event ``i``), int8 labels in
{+1 signal, -1 background} (section 1) and unit float32 weights.

Conventions shared by every workload:
  * values are drawn in float64 with ``numpy.random.default_rng`` (PCG64)
    and cast to float32;
  * the classes are exactly 50/50: the first half of the generation order is
    signal, then one seeded permutation shuffles events and labels together;
  * nothing here bins, boosts or scores: see ``oracle/`` and the library.
"""
from __future__ import annotations

import dataclasses
import hashlib

import numpy as np


@dataclasses.dataclass(frozen=True)
class ConfigSpec:
    """One workload: data shape, distribution family and fit hyper-parameters."""

    index: int
    name: str
    n_events: int
    n_features: int
    n_bins: int
    depth: int
    n_trees: int
    shrinkage: float
    subsample: float
    data_seed: int
    fit_seed: int
    family: str
    apply_events: int = 0      # fresh events for an apply-only workload
    apply_seed: int = 0


CONFIGS = {
    1: ConfigSpec(1, "toy 10k x 8, B=16, D=3, T=10", 10_000, 8, 16, 3, 10, 0.1, 0.5,
                  0, 0, "gauss_shift"),
    2: ConfigSpec(2, "fit 500k x 20, B=256, D=3, T=100", 500_000, 20, 256, 3, 100, 0.1, 0.5,
                  1, 1, "gauss_linspace"),
    3: ConfigSpec(3, "fit 2M x 40 correlated, B=256, D=3, T=200", 2_000_000, 40, 256, 3, 200,
                  0.1, 0.5, 2, 2, "one_factor"),
    4: ConfigSpec(4, "deep fit 10M x 40 mixed marginals, B=256, D=6, T=100", 10_000_000, 40,
                  256, 6, 100, 0.1, 0.5, 3, 3, "mixed"),
    5: ConfigSpec(5, "apply 400-tree D=3 forest to 50M x 40 fresh events", 2_000_000, 40, 256,
                  3, 400, 0.1, 0.5, 2, 4, "one_factor", apply_events=50_000_000,
                  apply_seed=4),
}


def _labels_signal_first(n: int) -> np.ndarray:
    y = np.full(n, -1, dtype=np.int8)
    y[: n // 2] = 1
    return y


def _one_factor_loadings(d: int) -> np.ndarray:
    # The loadings belong to the distribution, not to one sample of it: they
    # come from the training data seed of the correlated workload so that
    # fresh events for the apply workload share them.
    return np.random.default_rng(CONFIGS[3].data_seed).uniform(-0.7, 0.7, d)


def _gauss_shift(rng, n, d, n_sig):
    x = rng.standard_normal((d, n))
    x[: min(4, d), :n_sig] += 0.5
    return x


def _gauss_linspace(rng, n, d, n_sig):
    x = rng.standard_normal((d, n))
    k = min(10, d)
    x[:k, :n_sig] += np.linspace(0.1, 0.5, 10)[:k, None]
    return x


def _one_factor(rng, n, d, n_sig, lam):
    z = rng.standard_normal(n)
    e = rng.standard_normal((d, n))
    x = lam[:, None] * z[None, :] + np.sqrt(1.0 - lam * lam)[:, None] * e
    x[: min(20, d), :n_sig] += 0.3
    return x


_DISCRETE_LEVELS = (2, 3, 4, 5, 6, 8, 9, 10)


def _mixed_feature(rng, j, n, n_sig):
    """Feature j of the mixed-marginal workload (float64, generation order)."""
    if j <= 10:
        col = rng.standard_normal(n)
        if j <= 5:
            col[:n_sig] += 0.3
    elif j <= 21:
        col = rng.exponential(1.0, n)
        if j <= 16:
            col[:n_sig] *= 1.3
    elif j <= 31:
        col = rng.standard_cauchy(n)
        if j <= 25:
            col[:n_sig] += 0.3
    else:
        k = _DISCRETE_LEVELS[j - 32]
        col = np.empty(n)
        col[n_sig:] = rng.integers(0, k, n - n_sig)
        if j <= 35:
            p = 1.0 + 0.3 * np.arange(k) / (k - 1)
            col[:n_sig] = rng.choice(k, size=n_sig, p=p / p.sum())
        else:
            col[:n_sig] = rng.integers(0, k, n_sig)
    return col


def make_training_set(cfg: int | ConfigSpec, n_events: int | None = None):
    """Training events of one workload.

    ``n_events`` shrinks the sample (same distribution and seed) for parity
    cases that the oracle must finish in seconds.  Returns a dict with
    ``x`` float32 [d][n] (C-contiguous, feature-major), ``y`` int8 [n] and
    ``v`` float32 [n] (unit weights).
    """
    spec = CONFIGS[cfg] if isinstance(cfg, int) else cfg
    n = spec.n_events if n_events is None else int(n_events)
    d = spec.n_features
    n_sig = n // 2
    rng = np.random.default_rng(spec.data_seed)
    if spec.family == "gauss_shift":
        x64 = _gauss_shift(rng, n, d, n_sig)
    elif spec.family == "gauss_linspace":
        x64 = _gauss_linspace(rng, n, d, n_sig)
    elif spec.family == "one_factor":
        _ = rng.uniform(-0.7, 0.7, d)          # the loadings' draw, kept in the stream
        x64 = _one_factor(rng, n, d, n_sig, _one_factor_loadings(d))
    elif spec.family == "mixed":
        x = np.empty((d, n), dtype=np.float32)
        for j in range(d):
            x[j] = _mixed_feature(rng, j, n, n_sig)
        perm = rng.permutation(n)
        for j in range(d):
            x[j] = x[j][perm]
        y = _labels_signal_first(n)[perm]
        return {"x": x, "y": y, "v": np.ones(n, np.float32)}
    else:
        raise ValueError(spec.family)
    perm = rng.permutation(n)
    x = np.ascontiguousarray(x64[:, perm].astype(np.float32))
    y = _labels_signal_first(n)[perm]
    return {"x": x, "y": y, "v": np.ones(n, np.float32)}


def make_apply_chunk(chunk_index: int, chunk_events: int, cfg: int = 5):
    """One chunk of fresh events for the apply workload.

    Fresh events come from the correlated one-factor distribution of the
    training set.  Every chunk has its own seed ``[apply_seed, chunk_index]``
    so any chunk can be regenerated on its own.  Returns ``x`` float32 [d][m]
    and ``y`` int8 [m].
    """
    spec = CONFIGS[cfg]
    d = spec.n_features
    m = int(chunk_events)
    rng = np.random.default_rng([spec.apply_seed, int(chunk_index)])
    n_sig = m // 2
    x64 = _one_factor(rng, m, d, n_sig, _one_factor_loadings(d))
    perm = rng.permutation(m)
    x = np.ascontiguousarray(x64[:, perm].astype(np.float32))
    y = _labels_signal_first(m)[perm]
    return {"x": x, "y": y}


def _apply_chunk_x(args):
    cfg, index, m = args
    return make_apply_chunk(index, m, cfg)["x"]


def apply_chunks(n_events: int, chunk_events: int = 1_000_000, cfg: int = 5, workers: int = 16):
    """The first ``n_events`` fresh events of the apply workload as a stream.

    Yields ``(offset, x)`` in event order, ``x`` float32 [d][m] being chunk
    ``offset // chunk_events`` (the last one shortened), each drawn from its own
    seed exactly as ``make_apply_chunk`` draws it, with up to ``workers``
    processes drawing chunks ahead of the consumer.
    """
    import multiprocessing as mp

    n_chunks = (int(n_events) + chunk_events - 1) // chunk_events
    sizes = [min(chunk_events, int(n_events) - k * chunk_events) for k in range(n_chunks)]
    jobs = [(cfg, k, sizes[k]) for k in range(n_chunks)]
    if workers <= 1 or n_chunks <= 1:
        for k, job in enumerate(jobs):
            yield k * chunk_events, _apply_chunk_x(job)
        return
    ctx = mp.get_context("spawn")
    with ctx.Pool(min(workers, n_chunks)) as pool:
        for k, x in enumerate(pool.imap(_apply_chunk_x, jobs)):
            yield k * chunk_events, x


def random_binned(n: int, d: int, n_bins: int, seed: int, signal_fraction: float = 0.5):
    """Uniform random bin codes, labels and positive weights for unit tests."""
    rng = np.random.default_rng(seed)
    xb = rng.integers(0, n_bins, size=(d, n)).astype(np.uint8)
    y = np.where(rng.random(n) < signal_fraction, 1, -1).astype(np.int8)
    v = rng.uniform(0.5, 1.5, n).astype(np.float32)
    return xb, y, v


def random_forest(n_trees: int, depth: int, n_features: int, n_bins: int, seed: int):
    """A forest with random cuts and leaf values, for apply-only tests.

    Returns a dict of plain arrays in the library's model layout:
    ``cut_feature``/``cut_bin`` uint8 [T][2^D - 1] in heap order (node k at
    index k - 1), ``leaf`` float64 [T][2^D], ``f0`` float.
    """
    rng = np.random.default_rng(seed)
    n_inner = (1 << depth) - 1
    return {
        "cut_feature": rng.integers(0, n_features, (n_trees, n_inner)).astype(np.uint8),
        "cut_bin": rng.integers(1, max(2, n_bins), (n_trees, n_inner)).astype(np.uint8),
        "leaf": rng.normal(0.0, 0.05, (n_trees, 1 << depth)),
        "f0": float(rng.normal(0.0, 0.1)),
    }


def digest(*arrays) -> str:
    """SHA-256 over the raw bytes of the given arrays (dataset fingerprints)."""
    h = hashlib.sha256()
    for a in arrays:
        a = np.ascontiguousarray(a)
        h.update(str(a.dtype).encode())
        h.update(str(a.shape).encode())
        h.update(a.tobytes())
    return h.hexdigest()
