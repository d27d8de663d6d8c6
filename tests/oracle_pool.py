"""The oracle's binning of one feature, run in worker processes so that the
full-size parity cases bin tens of millions of values in seconds.  Each
worker calls the oracle's own functions unchanged, one feature at a time."""
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from oracle import fbdt_oracle as O  # noqa: E402


def bin_feature(args):
    column, n_bins = args
    b = O.quantile_boundaries(column, n_bins)
    return b, O.encode(column, b)


def bin_features_parallel(x, n_bins, workers=16):
    """Same result as the oracle's bin_features, feature by feature in a pool
    of spawned processes (none of them touches the GPU)."""
    import multiprocessing as mp
    import numpy as np
    with mp.get_context("spawn").Pool(min(workers, x.shape[0])) as pool:
        out = pool.map(bin_feature, [(x[j], n_bins) for j in range(x.shape[0])])
    return np.stack([b for b, _ in out]), np.stack([c for _, c in out])
