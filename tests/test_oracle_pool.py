"""The worker-pool binning used by the full-size parity cases is the
oracle's own binning (test infrastructure, not a pin of the oracle)."""
import numpy as np

from oracle import fbdt_oracle as O
from oracle_pool import bin_features_parallel
from synth import make_training_set


def test_parallel_oracle_binning_equals_serial():
    x = make_training_set(4, n_events=20_011)["x"]
    b1, c1 = O.bin_features(x, 256)
    b2, c2 = bin_features_parallel(x, 256, workers=2)
    assert np.array_equal(b1, b2) and np.array_equal(c1, c2)
