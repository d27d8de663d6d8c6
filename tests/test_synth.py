"""The seeded generators are deterministic and produce the stated shapes."""
import numpy as np

from synth import CONFIGS, digest, make_apply_chunk, make_training_set, random_forest


def test_training_sets_are_seeded_and_balanced():
    for idx in (1, 2, 3, 4):
        a = make_training_set(idx, n_events=2001 if idx > 1 else None)
        b = make_training_set(idx, n_events=2001 if idx > 1 else None)
        spec = CONFIGS[idx]
        n = a["x"].shape[1]
        assert a["x"].shape == (spec.n_features, n) and a["x"].dtype == np.float32
        assert a["x"].flags.c_contiguous
        assert digest(a["x"], a["y"]) == digest(b["x"], b["y"])
        assert int(np.sum(a["y"] > 0)) == n // 2 and set(np.unique(a["y"]).tolist()) == {-1, 1}
        assert np.all(a["v"] == 1.0)
        assert np.isfinite(a["x"]).all()


def test_mixed_workload_has_discrete_features():
    x = make_training_set(4, n_events=5000)["x"]
    for j, k in zip(range(32, 40), (2, 3, 4, 5, 6, 8, 9, 10)):
        assert len(np.unique(x[j])) == k


def test_apply_chunks_are_independent_and_reproducible():
    a = make_apply_chunk(3, 1000)
    b = make_apply_chunk(3, 1000)
    c = make_apply_chunk(4, 1000)
    assert np.array_equal(a["x"], b["x"]) and not np.array_equal(a["x"], c["x"])
    assert a["x"].shape == (40, 1000)


def test_random_forest_layout():
    f = random_forest(7, 3, 40, 256, 0)
    assert f["cut_feature"].shape == (7, 7) and f["cut_feature"].max() < 40
    assert f["cut_bin"].min() >= 1 and f["leaf"].shape == (7, 8)
