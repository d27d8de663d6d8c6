"""fbdt_best_cuts_noalloc against fbdt_best_cuts: the entry point for
callers that cannot allocate computes the same cuts from the same kernels
with its candidates in a fixed device array.  Two calls in a row, the second
on a smaller histogram, each compared bit for bit with the allocating call
on the same input."""
import numpy as np
import pytest
import torch

import paper_1609_06119_amd as fb

pytestmark = pytest.mark.gpu


def _hist(n_nodes, d, n_bins, seed):
    """Random float64 histograms [nodes][d][B][2] with empty bins, an empty
    node and a node whose every cut has gain 0 (one class only)."""
    rng = np.random.default_rng(seed)
    h = rng.exponential(1.0, (n_nodes, d, n_bins, 2))
    h[rng.random(h.shape[:3]) < 0.2] = 0.0
    h[0] = 0.0
    if n_nodes > 1:
        h[1, :, :, 1] = 0.0
    return torch.from_numpy(h).cuda()


def _noalloc(h):
    n_nodes = h.shape[0]
    f = torch.full((n_nodes,), 0xEE, dtype=torch.uint8, device="cuda")
    c = torch.full((n_nodes,), 0xEE, dtype=torch.uint8, device="cuda")
    g = torch.full((n_nodes,), np.nan, dtype=torch.float64, device="cuda")
    fb.best_cuts_noalloc(h, f, c, g)
    return f, c, g


def test_noalloc_best_cuts_equals_best_cuts_on_two_calls():
    big = _hist(64, 255, 256, 1)        # the largest shape the scratch holds
    small = _hist(5, 7, 33, 2)
    print("no-alloc best cuts: 64 x 255 x 256, then 5 x 7 x 33", flush=True)
    outs = [_noalloc(big), _noalloc(small)]      # back to back on the stream
    torch.cuda.synchronize()
    for h, (f, c, g) in zip((big, small), outs):
        rf, rc, rg = fb.best_cuts(h)
        torch.cuda.synchronize()
        assert torch.equal(f, rf) and torch.equal(c, rc)
        assert torch.equal(g, rg)               # bit for bit (no NaN among the gains)
        assert int(rf[0]) == 0 and int(rc[0]) == 1 and float(rg[0]) == 0.0   # empty node


def test_noalloc_best_cuts_rejects_bad_shapes_before_device_work():
    h = _hist(2, 3, 8, 3)
    with pytest.raises(fb.FbdtError) as ei:
        fb.best_cuts_noalloc(torch.zeros((65, 1, 2, 2), dtype=torch.float64, device="cuda"),
                             *[torch.empty(65, dtype=t, device="cuda")
                               for t in (torch.uint8, torch.uint8, torch.float64)])
    assert ei.value.status == "FBDT_E_INVAL"
    f, c, g = _noalloc(h)
    torch.cuda.synchronize()
    rf, rc, rg = fb.best_cuts(h)
    assert torch.equal(f, rf) and torch.equal(c, rc) and torch.equal(g, rg)
