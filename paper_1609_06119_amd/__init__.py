"""FastBDT's fit and apply hot path on AMD gfx950 (MI355X) through libfbdt.

Import is light: the HIP library is loaded on the first call.
"""
from .api import (  # noqa: F401
    Codes,
    FbdtError,
    Model,
    apply,
    apply_float,
    best_cuts,
    best_cuts_noalloc,
    bin,
    bin_transform,
    event_importance,
    feature_importance,
    fit,
    hist_timeline,
    histogram,
    leaf_values,
    padded_stride,
    reference_pass,
    route,
    set_option,
    timing_enable,
    timing_read,
    tree_weights,
)
from ._lib import EXPORTED, LIB_PATH, lib  # noqa: F401
