"""The C ABI library loads on the CPU host and exports every declared symbol."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fbdt.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fbdt_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("fbdt_bin", "fbdt_bin_transform", "fbdt_fit", "fbdt_apply",
                     "fbdt_model_export", "fbdt_model_import", "fbdt_model_free",
                     "fbdt_last_error", "fbdt_histogram", "fbdt_best_cuts", "fbdt_route",
                     "fbdt_tree_weights", "fbdt_leaf_values"):
        assert required in names


def test_library_exports_every_declared_symbol():
    from paper_1609_06119_amd._lib import EXPORTED, LIB_PATH
    if not os.path.exists(LIB_PATH):
        pytest.fail("libfbdt.so is not built (run __graft_entry__.build())")
    lib = ctypes.CDLL(LIB_PATH)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert missing == []
    assert sorted(EXPORTED) == declared_functions()


def test_argument_errors_need_no_device():
    # checks that run before any HIP call
    from paper_1609_06119_amd._lib import FitParams, lib
    L = lib()
    h = ctypes.c_void_p()
    p = FitParams(3, 10, 0.1, 0.5, 0)
    assert L.fbdt_fit(None, 10, 2, 16, 16, None, None, ctypes.byref(p), ctypes.byref(h), None,
                      None) == -1
    assert b"xb" in L.fbdt_last_error()
    buf = ctypes.create_string_buffer(64)
    aligned = (ctypes.addressof(buf) + 15) // 16 * 16
    assert L.fbdt_fit(ctypes.c_void_p(aligned), 10, 2, 15, 16, None, None, ctypes.byref(p),
                      ctypes.byref(h), None, None) == -1
    assert b"ldb" in L.fbdt_last_error()
    assert L.fbdt_set_option(b"no_such_option", 1) == -1
    assert L.fbdt_set_option(b"hist_threads", 100) == -1
    assert L.fbdt_set_option(b"hist_threads", 0) == 0
    # the histogram kernels are built for 1, 2, 4, 5 or 8 features per workgroup
    assert L.fbdt_set_option(b"hist_features_per_group", 3) == -1
    assert L.fbdt_set_option(b"hist_features_per_group", 5) == 0
    assert L.fbdt_set_option(b"hist_features_per_group", 0) == 0
    assert L.fbdt_set_option(b"hist_copies", 3) == -1
    assert L.fbdt_set_option(b"hist_copies", 4) == 0
    assert L.fbdt_set_option(b"hist_copies", 0) == 0
    # event lists below the root: auto, off or on; list passes are built for
    # 4, 8, 12, 20, 28 or 36 features per workgroup
    assert L.fbdt_set_option(b"hist_lists", 3) == -1
    assert L.fbdt_set_option(b"hist_lists", 0) == 0
    assert L.fbdt_set_option(b"list_features_per_group", 5) == -1
    assert L.fbdt_set_option(b"list_features_per_group", 20) == 0
    assert L.fbdt_set_option(b"list_features_per_group", 0) == 0
    assert L.fbdt_set_option(b"list_copies", 3) == -1
    assert L.fbdt_set_option(b"list_parts", 4097) == -1
    assert L.fbdt_set_option(b"list_parts", 0) == 0


def test_bench_refuses_more_than_one_gpu():
    """bench.py measures one GPU: --gpus 2 exits with status 2 and says so,
    before any device work."""
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stdout + r.stderr


def test_degenerate_arguments_are_rejected_before_device_work():
    """Empty and out-of-range inputs are FBDT_E_INVAL before any HIP call:
    no events, no or too many features, 1 or 257 bins, depth 0 or 8, no
    trees, shrinkage not finite and > 0, subsample outside (0, 1]."""
    from paper_1609_06119_amd._lib import FitParams, lib
    L = lib()
    h = ctypes.c_void_p()
    buf = ctypes.create_string_buffer(4096 + 16)
    xb = ctypes.c_void_p((ctypes.addressof(buf) + 15) // 16 * 16)
    y = ctypes.create_string_buffer(64)

    def fit(n=10, d=2, ldb=16, n_bins=16, params=(3, 10, 0.1, 0.5, 0)):
        p = FitParams(*params)
        return L.fbdt_fit(xb, n, d, ldb, n_bins, y, None, ctypes.byref(p), ctypes.byref(h),
                          None, None)

    for kw, needle in [(dict(n=0), b"n = 0"), (dict(d=0), b"d = 0"), (dict(d=256), b"d = 256"),
                       (dict(n_bins=1), b"n_bins"), (dict(n_bins=257), b"n_bins"),
                       (dict(params=(0, 10, 0.1, 0.5, 0)), b"depth"),
                       (dict(params=(8, 10, 0.1, 0.5, 0)), b"depth"),
                       (dict(params=(3, 0, 0.1, 0.5, 0)), b"n_trees"),
                       (dict(params=(3, 10, 0.0, 0.5, 0)), b"shrinkage"),
                       (dict(params=(3, 10, float("inf"), 0.5, 0)), b"shrinkage"),
                       (dict(params=(3, 10, 0.1, 0.0, 0)), b"subsample"),
                       (dict(params=(3, 10, 0.1, 1.5, 0)), b"subsample")]:
        assert fit(**kw) == -1, kw
        assert needle in L.fbdt_last_error(), (kw, L.fbdt_last_error())
