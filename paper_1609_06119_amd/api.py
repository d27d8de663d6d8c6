"""Python binding of libfbdt: argument marshalling only.

Every step of binning, fitting and applying runs in the HIP library; this
module checks tensor shapes and dtypes, passes device pointers and the
current HIP stream, and turns error codes into exceptions.  PyTorch serves
as the device allocator and stream provider.
"""
from __future__ import annotations

import ctypes as C
import dataclasses

import numpy as np
import torch

from ._lib import FitParams, FbdtError, KERNEL_KINDS, ModelView, check, lib

__all__ = ["Codes", "Model", "bin", "bin_transform", "fit", "apply", "tree_weights",
           "histogram", "best_cuts", "best_cuts_noalloc", "route", "leaf_values",
           "timing_enable", "timing_read", "set_option", "hist_timeline", "reference_pass",
           "FbdtError", "padded_stride"]


def padded_stride(n: int) -> int:
    """Row stride of a code buffer: n rounded up to a multiple of 64 bytes."""
    return (int(n) + 63) // 64 * 64


def _stream():
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t: torch.Tensor | None):
    return C.c_void_p(t.data_ptr()) if t is not None else None


def _need(t: torch.Tensor, dtype, name: str, numel: int | None = None):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if numel is not None and t.numel() < numel:
        raise ValueError(f"{name} holds {t.numel()} elements, needs {numel}")


@dataclasses.dataclass
class Codes:
    """Binned features: uint8 [d][ldb] on the device, first n columns valid."""

    data: torch.Tensor
    n: int

    @property
    def d(self) -> int:
        return int(self.data.shape[0])

    @property
    def ldb(self) -> int:
        return int(self.data.stride(0))

    @staticmethod
    def empty(d: int, n: int, device="cuda") -> "Codes":
        return Codes(torch.zeros((d, padded_stride(n)), dtype=torch.uint8, device=device), int(n))

    @staticmethod
    def from_numpy(xb: np.ndarray, device="cuda") -> "Codes":
        xb = np.asarray(xb, dtype=np.uint8)
        d, n = xb.shape
        host = np.zeros((d, padded_stride(n)), np.uint8)
        host[:, :n] = xb
        return Codes(torch.from_numpy(host).to(device), n)

    def numpy(self) -> np.ndarray:
        return self.data[:, : self.n].cpu().numpy()


class Model:
    """A fitted forest owned by libfbdt (heap order: node k at index k - 1)."""

    def __init__(self, handle: C.c_void_p):
        self._h = handle

    @property
    def handle(self):
        return self._h

    def __del__(self):
        h, self._h = getattr(self, "_h", None), None
        if h and lib is not None:
            try:
                lib().fbdt_model_free(h)
            except Exception:
                pass

    def export(self) -> dict:
        """Copies of the model arrays (numpy)."""
        v = ModelView()
        check("fbdt_model_export", lib().fbdt_model_export(self._h, C.byref(v)))
        T, D = v.n_trees, v.depth
        nin, nleaf = (1 << D) - 1, 1 << D

        def arr(p, count, dt):
            return np.ctypeslib.as_array(p, shape=(count,)).astype(dt, copy=True)

        out = {
            "n_trees": T, "depth": D, "n_features": v.n_features, "n_bins": v.n_bins,
            "f0": float(v.f0),
            "cut_feature": arr(v.cut_feature, T * nin, np.uint8).reshape(T, nin),
            "cut_bin": arr(v.cut_bin, T * nin, np.uint8).reshape(T, nin),
            "gain": arr(v.gain, T * nin, np.float64).reshape(T, nin),
            "leaf": arr(v.leaf, T * nleaf, np.float64).reshape(T, nleaf),
        }
        if v.boundaries:
            out["boundaries"] = arr(v.boundaries, v.n_features * (v.n_bins - 1),
                                    np.float32).reshape(v.n_features, v.n_bins - 1)
        if v.inner:   # missing values: boost weights of the inner nodes
            out["inner"] = arr(v.inner, T * nin, np.float64).reshape(T, nin)
        return out

    def set_boundaries(self, boundaries) -> "Model":
        """Attach the training bin boundaries [d][B-1] (for apply_float)."""
        b = np.ascontiguousarray(boundaries, np.float32)
        check("fbdt_model_set_boundaries",
              lib().fbdt_model_set_boundaries(self._h, b.ctypes.data_as(C.c_void_p)))
        return self

    @staticmethod
    def from_arrays(cut_feature, cut_bin, leaf, f0: float, n_features: int, n_bins: int,
                    gain=None, boundaries=None, inner=None) -> "Model":
        cf = np.ascontiguousarray(cut_feature, np.uint8)
        cb = np.ascontiguousarray(cut_bin, np.uint8)
        lf = np.ascontiguousarray(leaf, np.float64)
        T, nin = cf.shape
        D = int(np.log2(nin + 1))
        if (1 << D) - 1 != nin or lf.shape != (T, 1 << D) or cb.shape != cf.shape:
            raise ValueError("inconsistent forest arrays")
        keep = [cf, cb, lf]
        v = ModelView()
        v.n_trees, v.depth, v.n_features, v.n_bins, v.f0 = T, D, int(n_features), int(n_bins), float(f0)
        v.cut_feature = cf.ctypes.data_as(C.POINTER(C.c_uint8))
        v.cut_bin = cb.ctypes.data_as(C.POINTER(C.c_uint8))
        v.leaf = lf.ctypes.data_as(C.POINTER(C.c_double))
        if gain is not None:
            g = np.ascontiguousarray(gain, np.float64)
            keep.append(g)
            v.gain = g.ctypes.data_as(C.POINTER(C.c_double))
        if boundaries is not None:
            b = np.ascontiguousarray(boundaries, np.float32)
            keep.append(b)
            v.boundaries = b.ctypes.data_as(C.POINTER(C.c_float))
        if inner is not None:
            iv = np.ascontiguousarray(inner, np.float64)
            if iv.shape != cf.shape:
                raise ValueError("inner must have the shape of cut_feature")
            keep.append(iv)
            v.inner = iv.ctypes.data_as(C.POINTER(C.c_double))
        h = C.c_void_p()
        check("fbdt_model_import", lib().fbdt_model_import(C.byref(v), C.byref(h)))
        del keep
        return Model(h)


def bin(x: torch.Tensor, n_bins: int, codes: Codes | None = None):
    """Equal-frequency binning of a feature-major float32 sample x [d][n]
    (row stride x.stride(0)).  Returns (boundaries numpy float32 [d][B-1], Codes)."""
    _need_rows(x)
    d, n = int(x.shape[0]), int(x.shape[1])
    codes = codes or Codes.empty(d, n, x.device)
    bounds = np.zeros((d, n_bins - 1), np.float32)
    check("fbdt_bin", lib().fbdt_bin(_ptr(x), n, d, _row_stride(x), n_bins,
                                     bounds.ctypes.data_as(C.c_void_p), _ptr(codes.data),
                                     codes.ldb, _stream()))
    return bounds, codes


def _need_rows(x: torch.Tensor):
    if not isinstance(x, torch.Tensor) or not x.is_cuda or x.dtype != torch.float32:
        raise TypeError("x must be a float32 CUDA (HIP) tensor [d][n]")
    if x.dim() != 2 or (x.stride(1) != 1 and x.shape[1] > 1):
        raise ValueError("x must be 2-D [d][n] with unit stride along events")


def _row_stride(x: torch.Tensor) -> int:
    """Elements between feature rows; a single row may report any stride."""
    return int(x.stride(0)) if x.shape[0] > 1 else int(x.shape[1])


def bin_transform(x: torch.Tensor, boundaries: np.ndarray, codes: Codes | None = None) -> Codes:
    """Bin fresh events with training boundaries [d][B-1]."""
    _need_rows(x)
    d, n = int(x.shape[0]), int(x.shape[1])
    b = np.ascontiguousarray(boundaries, np.float32)
    if b.shape[0] != d:
        raise ValueError("boundaries must have one row per feature")
    codes = codes or Codes.empty(d, n, x.device)
    check("fbdt_bin_transform",
          lib().fbdt_bin_transform(_ptr(x), n, d, _row_stride(x), b.shape[1] + 1,
                                   b.ctypes.data_as(C.c_void_p), _ptr(codes.data), codes.ldb,
                                   _stream()))
    return codes


def fit(codes: Codes, y: torch.Tensor, n_bins: int, depth: int, n_trees: int,
        shrinkage: float = 0.1, subsample: float = 0.5, seed: int = 0,
        w: torch.Tensor | None = None, score_out: torch.Tensor | None = None) -> Model:
    """Fit a forest on binned features; y int8 [n] in {+1, -1}, w float32 [n] or None."""
    n = codes.n
    _need(y, torch.int8, "y", n)
    if w is not None:
        _need(w, torch.float32, "w", n)
    if score_out is not None:
        _need(score_out, torch.float64, "score_out", n)
    p = FitParams(int(depth), int(n_trees), float(shrinkage), float(subsample),
                  int(seed) & 0xFFFFFFFFFFFFFFFF)
    h = C.c_void_p()
    check("fbdt_fit", lib().fbdt_fit(_ptr(codes.data), n, codes.d, codes.ldb, int(n_bins),
                                     _ptr(y), _ptr(w), C.byref(p), C.byref(h), _ptr(score_out),
                                     _stream()))
    return Model(h)


def apply(model: Model, codes: Codes, prob: torch.Tensor | None = None,
          score: torch.Tensor | None = None) -> torch.Tensor:
    """P(signal) float32 [n] of binned events (score float64 [n] optionally)."""
    n = codes.n
    prob = prob if prob is not None else torch.empty(n, dtype=torch.float32,
                                                     device=codes.data.device)
    _need(prob, torch.float32, "prob", n)
    if score is not None:
        _need(score, torch.float64, "score", n)
    check("fbdt_apply", lib().fbdt_apply(model.handle, _ptr(codes.data), n, codes.d, codes.ldb,
                                         _ptr(prob), _ptr(score), _stream()))
    return prob


def apply_float(model: Model, x: torch.Tensor, prob: torch.Tensor | None = None,
                score: torch.Tensor | None = None) -> torch.Tensor:
    """P(signal) float32 [n] of float32 events x [d][n] (row stride x.stride(0)),
    tested against the model's value thresholds; score float64 [n] optionally."""
    _need_rows(x)
    d, n = int(x.shape[0]), int(x.shape[1])
    prob = prob if prob is not None else torch.empty(n, dtype=torch.float32, device=x.device)
    _need(prob, torch.float32, "prob", n)
    if score is not None:
        _need(score, torch.float64, "score", n)
    check("fbdt_apply_float", lib().fbdt_apply_float(model.handle, _ptr(x), n, d, _row_stride(x),
                                                     _ptr(prob), _ptr(score), _stream()))
    return prob


def feature_importance(model: Model) -> np.ndarray:
    """Summed separation gain per feature over every node of every tree."""
    n_features = model.export()["n_features"]
    out = np.zeros(n_features, np.float64)
    check("fbdt_feature_importance",
          lib().fbdt_feature_importance(model.handle, out.ctypes.data_as(C.c_void_p)))
    return out


def event_importance(model: Model, codes: Codes, out: torch.Tensor | None = None) -> torch.Tensor:
    """Per-event importance float64 [d][n]: the gains on each event's path,
    summed per cut feature."""
    n, d = codes.n, codes.d
    out = out if out is not None else torch.empty((d, n), dtype=torch.float64,
                                                  device=codes.data.device)
    if out.dtype != torch.float64 or out.dim() != 2 or out.shape[0] != d or out.shape[1] < n \
            or out.stride(1) != 1 or not out.is_cuda:
        raise ValueError("out must be a float64 CUDA tensor [d][>= n] with unit stride along events")
    check("fbdt_event_importance",
          lib().fbdt_event_importance(model.handle, _ptr(codes.data), n, d, codes.ldb, _ptr(out),
                                      out.stride(0), _stream()))
    return out


def tree_weights(y, v, F, seed: int, tree: int, alpha: float, w_out=None) -> torch.Tensor:
    n = int(y.numel())
    _need(y, torch.int8, "y")
    _need(F, torch.float64, "F", n)
    if v is not None:
        _need(v, torch.float32, "v", n)
    w_out = w_out if w_out is not None else torch.empty(n, dtype=torch.float32, device=y.device)
    check("fbdt_tree_weights", lib().fbdt_tree_weights(_ptr(y), _ptr(v), _ptr(F), n,
                                                       int(seed) & 0xFFFFFFFFFFFFFFFF,
                                                       int(tree), float(alpha), _ptr(w_out),
                                                       _stream()))
    return w_out


def histogram(codes: Codes, node: torch.Tensor, w: torch.Tensor, layer: int,
              n_bins: int) -> torch.Tensor:
    n = codes.n
    _need(node, torch.uint8, "node", n)
    _need(w, torch.float32, "w", n)
    hist = torch.empty(((1 << layer), codes.d, n_bins, 2), dtype=torch.float64,
                       device=codes.data.device)
    check("fbdt_histogram", lib().fbdt_histogram(_ptr(codes.data), n, codes.d, codes.ldb,
                                                 int(n_bins), _ptr(node), _ptr(w), int(layer),
                                                 _ptr(hist), _stream()))
    return hist


def best_cuts(hist: torch.Tensor):
    _need(hist, torch.float64, "hist")
    n_nodes, d, n_bins, two = hist.shape
    if two != 2:
        raise ValueError("hist must be [nodes][d][B][2]")
    dev = hist.device
    f = torch.empty(n_nodes, dtype=torch.uint8, device=dev)
    c = torch.empty(n_nodes, dtype=torch.uint8, device=dev)
    g = torch.empty(n_nodes, dtype=torch.float64, device=dev)
    check("fbdt_best_cuts", lib().fbdt_best_cuts(_ptr(hist), n_nodes, d, n_bins, _ptr(f),
                                                 _ptr(c), _ptr(g), _stream()))
    return f, c, g


def best_cuts_noalloc(hist: torch.Tensor, cut_feature: torch.Tensor, cut_bin: torch.Tensor,
                      gain: torch.Tensor):
    """fbdt_best_cuts_noalloc into caller-allocated outputs (uint8, uint8,
    float64, one entry per node); stream-ordered, allocates nothing."""
    _need(hist, torch.float64, "hist")
    n_nodes, d, n_bins, two = hist.shape
    if two != 2:
        raise ValueError("hist must be [nodes][d][B][2]")
    _need(cut_feature, torch.uint8, "cut_feature", n_nodes)
    _need(cut_bin, torch.uint8, "cut_bin", n_nodes)
    _need(gain, torch.float64, "gain", n_nodes)
    check("fbdt_best_cuts_noalloc",
          lib().fbdt_best_cuts_noalloc(_ptr(hist), n_nodes, d, n_bins, _ptr(cut_feature),
                                       _ptr(cut_bin), _ptr(gain), _stream()))


def route(codes: Codes, node: torch.Tensor, cut_feature: torch.Tensor, cut_bin: torch.Tensor,
          layer: int) -> torch.Tensor:
    n = codes.n
    _need(node, torch.uint8, "node", n)
    _need(cut_feature, torch.uint8, "cut_feature", 1 << layer)
    _need(cut_bin, torch.uint8, "cut_bin", 1 << layer)
    check("fbdt_route", lib().fbdt_route(_ptr(codes.data), n, codes.d, codes.ldb, _ptr(node),
                                         _ptr(cut_feature), _ptr(cut_bin), int(layer),
                                         _stream()))
    return node


def leaf_values(node, y, v, F, depth: int, seed: int, tree: int, alpha: float,
                eta: float) -> torch.Tensor:
    n = int(node.numel())
    _need(node, torch.uint8, "node")
    _need(y, torch.int8, "y", n)
    _need(F, torch.float64, "F", n)
    if v is not None:
        _need(v, torch.float32, "v", n)
    leaf = torch.empty(1 << depth, dtype=torch.float64, device=node.device)
    check("fbdt_leaf_values", lib().fbdt_leaf_values(_ptr(node), _ptr(y), _ptr(v), _ptr(F), n,
                                                     int(depth), int(seed) & 0xFFFFFFFFFFFFFFFF,
                                                     int(tree), float(alpha), float(eta),
                                                     _ptr(leaf), _stream()))
    return leaf


def timing_enable(kinds=("histogram",)):
    """Time every launch of the given kernel kinds (an empty tuple: off)."""
    mask = 0
    for k in kinds:
        mask |= 1 << KERNEL_KINDS[k]
    check("fbdt_timing_enable", lib().fbdt_timing_enable(mask))


def timing_read(kind: str):
    """(launches, total milliseconds, algorithmic bytes) of one kernel kind."""
    k = C.c_int64()
    ms = C.c_double()
    by = C.c_double()
    check("fbdt_timing_read", lib().fbdt_timing_read(KERNEL_KINDS[kind], C.byref(k),
                                                     C.byref(ms), C.byref(by)))
    return int(k.value), float(ms.value), float(by.value)


def hist_timeline():
    """Phase timeline of the histogram launches of the last fit made with
    option hist_timeline = 1: (stamps uint64 [launches][max_blocks][8],
    blocks int32 [launches], clock rate in kHz); None if there was none."""
    launches, mb, rate = C.c_int64(), C.c_int32(), C.c_int64()
    blocks = C.POINTER(C.c_int32)()
    stamps = C.POINTER(C.c_uint64)()
    check("fbdt_hist_timeline", lib().fbdt_hist_timeline(C.byref(launches), C.byref(mb),
                                                          C.byref(blocks), C.byref(stamps),
                                                          C.byref(rate)))
    if launches.value == 0:
        return None
    k, m = launches.value, mb.value
    st = np.ctypeslib.as_array(stamps, shape=(k * m * 8,)).reshape(k, m, 8).copy()
    bl = np.ctypeslib.as_array(blocks, shape=(k,)).copy()
    return st, bl, rate.value


def reference_pass(kind: int, codes: Codes, n_bins: int, layer: int, w: torch.Tensor,
                   node: torch.Tensor | None = None):
    """fbdt_reference_pass: kind 0 (empty) or 1 (read only) on the histogram
    pass's launch shape for `layer`; w float32 and node uint8 padded to a
    multiple of 8 events."""
    npad = (codes.n + 7) // 8 * 8
    _need(w, torch.float32, "w", npad)
    if node is not None:
        _need(node, torch.uint8, "node", npad)
    check("fbdt_reference_pass",
          lib().fbdt_reference_pass(int(kind), _ptr(codes.data), codes.n, codes.d, codes.ldb,
                                    int(n_bins), int(layer), _ptr(node), _ptr(w), _stream()))


def set_option(name: str, value: int):
    check("fbdt_set_option", lib().fbdt_set_option(name.encode(), int(value)))
