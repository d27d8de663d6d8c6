"""Drives the host runtime's argument checks and host-only calls of a libfbdt
build (path in argv[1]) through the C ABI; run by test_host_sanitizers.py in
a process with the AddressSanitizer runtime preloaded.  No call here reaches
the device: every one either fails its argument checks or works on host
memory only (model import / export / importance / free, options, timing
tallies, the error message).  Prints "sanitizer driver: N checks ok"."""
import ctypes as C
import sys

import numpy as np

sys.path.insert(0, sys.argv[2])
from paper_1609_06119_amd._lib import FitParams, ModelView, _declare  # noqa: E402

L = C.CDLL(sys.argv[1])
_declare(L)
INVAL, SHAPE = -1, -5
checks = 0


def expect(rc, code, word=None):
    global checks
    assert rc == code, (rc, code, L.fbdt_last_error())
    if word is not None:
        assert word.encode() in L.fbdt_last_error(), (word, L.fbdt_last_error())
    checks += 1


buf = C.create_string_buffer(4096 + 16)
a16 = C.c_void_p((C.addressof(buf) + 15) // 16 * 16)
odd = C.c_void_p(a16.value + 1)
out = C.c_void_p()
p = FitParams(3, 10, 0.1, 0.5, 0)

# fbdt_fit
expect(L.fbdt_fit(None, 10, 2, 16, 16, a16, None, C.byref(p), C.byref(out), None, None), INVAL, "xb")
expect(L.fbdt_fit(a16, 0, 2, 16, 16, a16, None, C.byref(p), C.byref(out), None, None), INVAL, "n =")
expect(L.fbdt_fit(a16, 10, 0, 16, 16, a16, None, C.byref(p), C.byref(out), None, None), INVAL, "d =")
expect(L.fbdt_fit(a16, 10, 256, 16, 16, a16, None, C.byref(p), C.byref(out), None, None), INVAL, "d =")
expect(L.fbdt_fit(a16, 10, 2, 15, 16, a16, None, C.byref(p), C.byref(out), None, None), INVAL, "ldb")
expect(L.fbdt_fit(odd, 10, 2, 16, 16, a16, None, C.byref(p), C.byref(out), None, None), INVAL, "aligned")
expect(L.fbdt_fit(a16, 10, 2, 16, 1, a16, None, C.byref(p), C.byref(out), None, None), INVAL, "n_bins")
expect(L.fbdt_fit(a16, 10, 2, 16, 257, a16, None, C.byref(p), C.byref(out), None, None), INVAL, "n_bins")
expect(L.fbdt_fit(a16, 10, 2, 16, 16, None, None, C.byref(p), C.byref(out), None, None), INVAL, "y")
expect(L.fbdt_fit(a16, 10, 2, 16, 16, a16, None, None, C.byref(out), None, None), INVAL, "params")
expect(L.fbdt_fit(a16, 10, 2, 16, 16, a16, None, C.byref(p), None, None, None), INVAL, "out")
for bad in (FitParams(0, 10, 0.1, 0.5, 0), FitParams(8, 10, 0.1, 0.5, 0), FitParams(3, 0, 0.1, 0.5, 0),
            FitParams(3, 10, 0.0, 0.5, 0), FitParams(3, 10, float("inf"), 0.5, 0),
            FitParams(3, 10, float("nan"), 0.5, 0), FitParams(3, 10, 0.1, 0.0, 0),
            FitParams(3, 10, 0.1, 1.5, 0), FitParams(3, 10, 0.1, float("nan"), 0)):
    expect(L.fbdt_fit(a16, 10, 2, 16, 16, a16, None, C.byref(bad), C.byref(out), None, None), INVAL)

# binning
expect(L.fbdt_bin(None, 10, 2, 10, 16, a16, a16, 16, None), INVAL, "x")
expect(L.fbdt_bin(a16, 10, 2, 9, 16, a16, a16, 16, None), INVAL, "ldx")
expect(L.fbdt_bin(a16, 10, 2, 10, 16, None, a16, 16, None), INVAL, "boundaries")
expect(L.fbdt_bin_transform(a16, 10, 2, 10, 16, None, a16, 16, None), INVAL, "boundaries")
bnd = np.zeros((2, 15), np.float32)
bnd[1, 3] = -1.0
expect(L.fbdt_bin_transform(a16, 10, 2, 10, 16, bnd.ctypes.data_as(C.c_void_p), a16, 16, None),
       INVAL, "ascending")

# apply, importance, single steps
expect(L.fbdt_apply(None, a16, 10, 2, 16, a16, None, None), INVAL, "model")
expect(L.fbdt_apply_float(None, a16, 10, 2, 16, a16, None, None), INVAL, "model")
expect(L.fbdt_event_importance(None, a16, 10, 2, 16, a16, 16, None), INVAL, "model")
expect(L.fbdt_tree_weights(None, None, None, 10, 0, 0, 0.5, None, None), INVAL)
expect(L.fbdt_tree_weights(a16, None, a16, 0, 0, 0, 0.5, a16, None), INVAL)
expect(L.fbdt_tree_weights(a16, None, a16, 10, 0, -1, 0.5, a16, None), INVAL)
expect(L.fbdt_tree_weights(a16, None, a16, 10, 0, 0, 0.0, a16, None), INVAL)
expect(L.fbdt_histogram(a16, 10, 2, 16, 16, None, a16, 0, a16, None), INVAL)
expect(L.fbdt_histogram(a16, 10, 2, 16, 16, odd, a16, 0, a16, None), INVAL, "aligned")
expect(L.fbdt_histogram(a16, 10, 2, 16, 16, a16, a16, 7, a16, None), INVAL, "layer")
expect(L.fbdt_best_cuts(None, 1, 2, 16, a16, a16, a16, None), INVAL)
expect(L.fbdt_best_cuts(a16, 65, 2, 16, a16, a16, a16, None), INVAL, "n_nodes")
expect(L.fbdt_best_cuts(odd, 1, 2, 16, a16, a16, a16, None), INVAL, "aligned")
expect(L.fbdt_best_cuts_noalloc(a16, 0, 2, 16, a16, a16, a16, None), INVAL, "n_nodes")
expect(L.fbdt_best_cuts_noalloc(a16, 1, 256, 16, a16, a16, a16, None), INVAL, "d not")
expect(L.fbdt_best_cuts_noalloc(a16, 1, 2, 1, a16, a16, a16, None), INVAL, "n_bins")
expect(L.fbdt_route(a16, 10, 2, 16, None, a16, a16, 0, None), INVAL)
expect(L.fbdt_route(a16, 10, 2, 16, a16, a16, a16, 7, None), INVAL, "layer")
expect(L.fbdt_leaf_values(None, a16, None, a16, 10, 3, 0, 0, 0.5, 0.1, a16, None), INVAL)
expect(L.fbdt_leaf_values(a16, a16, None, a16, 10, 8, 0, 0, 0.5, 0.1, a16, None), INVAL, "depth")
expect(L.fbdt_reference_pass(3, a16, 10, 2, 16, 16, 0, None, a16, None), INVAL, "kind")
expect(L.fbdt_reference_pass(0, a16, 10, 2, 16, 16, 0, None, None, None), INVAL, "w")

# options and timing tallies (host only)
expect(L.fbdt_set_option(None, 0), INVAL)
expect(L.fbdt_set_option(b"no_such_option", 1), INVAL, "unknown")
expect(L.fbdt_set_option(b"hist_threads", 100), INVAL)
expect(L.fbdt_set_option(b"hist_features_per_group", 3), INVAL)
expect(L.fbdt_set_option(b"hist_copies", 3), INVAL)
expect(L.fbdt_set_option(b"apply_threads", 2048), INVAL)
expect(L.fbdt_set_option(b"fit_graphs", -1), INVAL)
expect(L.fbdt_set_option(b"hist_lists", 3), INVAL)
expect(L.fbdt_set_option(b"list_features_per_group", 16), INVAL)
expect(L.fbdt_set_option(b"list_parts", 5000), INVAL)
expect(L.fbdt_set_option(b"list_copies", 8), INVAL)
for name in (b"hist_features_per_group", b"hist_event_chunks", b"hist_threads", b"hist_copies",
             b"apply_threads", b"hist_timeline", b"fail_alloc", b"hist_lists",
             b"list_features_per_group", b"list_parts", b"list_copies"):
    expect(L.fbdt_set_option(name, 0), 0)
expect(L.fbdt_set_option(b"fit_graphs", 1), 0)
expect(L.fbdt_timing_enable(0), 0)
k, ms, by = C.c_int64(), C.c_double(), C.c_double()
expect(L.fbdt_timing_read(8, C.byref(k), C.byref(ms), C.byref(by)), INVAL, "kind")
expect(L.fbdt_timing_read(0, C.byref(k), C.byref(ms), C.byref(by)), 0)
assert k.value == 0
nl, mb, rate = C.c_int64(), C.c_int32(), C.c_int64()
bl, st = C.POINTER(C.c_int32)(), C.POINTER(C.c_uint64)()
expect(L.fbdt_hist_timeline(None, C.byref(mb), C.byref(bl), C.byref(st), C.byref(rate)), INVAL)
expect(L.fbdt_hist_timeline(C.byref(nl), C.byref(mb), C.byref(bl), C.byref(st), C.byref(rate)), 0)
assert nl.value == 0

# model import / export / importance / free (host memory only)
T, D, d, B = 5, 3, 4, 16
rng = np.random.default_rng(0)
cf = rng.integers(0, d, (T, 7)).astype(np.uint8)
cb = rng.integers(1, B, (T, 7)).astype(np.uint8)
gn = rng.random((T, 7))
lf = rng.normal(size=(T, 8))
bd = np.sort(rng.normal(size=(d, B - 1)).astype(np.float32), axis=1)


def view(**kw):
    v = ModelView(T, D, d, B, 0.25, cf.ctypes.data_as(C.POINTER(C.c_uint8)),
                  cb.ctypes.data_as(C.POINTER(C.c_uint8)), gn.ctypes.data_as(C.POINTER(C.c_double)),
                  lf.ctypes.data_as(C.POINTER(C.c_double)),
                  bd.ctypes.data_as(C.POINTER(C.c_float)), None)
    for key, val in kw.items():
        setattr(v, key, val)
    return v


expect(L.fbdt_model_import(None, C.byref(out)), INVAL)
for bad in (dict(n_trees=0), dict(depth=8), dict(n_features=256), dict(n_bins=1),
            dict(n_bins=257), dict(cut_feature=None), dict(leaf=None), dict(f0=float("nan"))):
    expect(L.fbdt_model_import(C.byref(view(**bad)), C.byref(out)), INVAL)
cf[0, 0] = d
expect(L.fbdt_model_import(C.byref(view()), C.byref(out)), INVAL, "cut feature")
cf[0, 0] = 0
cb[0, 0] = B
expect(L.fbdt_model_import(C.byref(view()), C.byref(out)), INVAL, "cut bin")
cb[0, 0] = 1
bd[1, 2] = np.nan
expect(L.fbdt_model_import(C.byref(view()), C.byref(out)), INVAL, "NaN")
bd[1, 2] = bd[1, 1]
inner = np.zeros((T, 7))
v = view()
v.inner = inner.ctypes.data_as(C.POINTER(C.c_double))
v.n_bins = 256
expect(L.fbdt_model_import(C.byref(v), C.byref(out)), INVAL)
expect(L.fbdt_model_import(C.byref(view()), C.byref(out)), 0)
m = out
ev = ModelView()
expect(L.fbdt_model_export(None, C.byref(ev)), INVAL)
expect(L.fbdt_model_export(m, C.byref(ev)), 0)
assert ev.n_trees == T and ev.f0 == 0.25 and ev.cut_bin[3] == cb.reshape(-1)[3]
imp = np.zeros(d)
expect(L.fbdt_feature_importance(m, imp.ctypes.data_as(C.c_void_p)), 0)
ref = np.zeros(d)
np.add.at(ref, cf.reshape(-1), gn.reshape(-1))
assert np.allclose(imp, ref, rtol=1e-12)
expect(L.fbdt_feature_importance(None, imp.ctypes.data_as(C.c_void_p)), INVAL)
expect(L.fbdt_model_set_boundaries(m, None), INVAL)
bad_b = bd.copy()
bad_b[0] = bad_b[0][::-1].copy()   # descending
expect(L.fbdt_model_set_boundaries(m, bad_b.ctypes.data_as(C.c_void_p)), INVAL, "ascending")
expect(L.fbdt_apply(m, a16, 10, 2, 16, a16, None, None), SHAPE)
expect(L.fbdt_apply_float(m, a16, 10, 2, 16, a16, None, None), SHAPE)
expect(L.fbdt_event_importance(m, a16, 10, 4, 16, a16, 9, None), INVAL, "ldi")
L.fbdt_model_free(m)
L.fbdt_model_free(None)
print(f"sanitizer driver: {checks} checks ok", flush=True)
