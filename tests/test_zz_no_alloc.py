"""The allocation-free weight gradient (dc_conv_bwd_filter_noalloc) against
the entry point it mirrors (dc_conv_bwd_filter with a caller workspace):
identical bits on two calls in a row, the second on a smaller problem, so
that the fixed device workspace is reused with a different layout of
partials.  Both go through the C ABI."""
import numpy as np
import pytest
import torch

import harness as H
import paper_1903_06681_amd as dc
import workloads as wl

pytestmark = pytest.mark.gpu

X, DY, ALL = dc.DC_X, dc.DC_DY, dc.DC_ALL_TILES


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()


def _bits(t):
    return t.view(torch.int32)


def _inputs(L, tile):
    p = dc.Problem.of(L)
    nt = L.P * L.Q
    x, dy = wl.draw(L, "x"), wl.draw(L, "dy")
    xt = H.alloc_tiles(p, X, nt, L.dtype)
    dyt = H.alloc_tiles(p, DY, nt, L.dtype)
    H.scatter_interiors(xt, H.to_device(x, L.dtype), p, X)
    H.scatter_interiors(dyt, H.to_device(dy, L.dtype), p, DY)
    H.fill_halos_all_tiles(p, X, xt, L.dtype)
    H.fill_halos_all_tiles(p, DY, dyt, L.dtype)
    if tile == ALL:
        return p, xt, dyt
    return p, xt[tile].clone(), dyt[tile].clone()


# (layer, tile, accumulate): the benchmark's c5a tile (k-slice kernel, 9 MiB
# of partials), then smaller problems on other kernels
CASES = [
    (wl.LAYERS["c5a"], 5, 0),
    (wl.small("c5a", N=2, H=96, W=96, P=3, Q=3), ALL, 0),
    (wl.small("c5b", N=2, H=72, W=72, P=2, Q=2), 1, 1),
    (wl.LAYERS["c2"], ALL, 0),
]


def test_noalloc_equals_workspace_entry_point_on_consecutive_calls():
    for L, tile, acc in CASES:
        print(f"[noalloc] {L.name} tile {tile} accumulate {acc}", flush=True)
        p, xp, dyp = _inputs(L, tile)
        need = dc.bwd_filter_workspace_bytes(p, tile)
        assert 0 < need <= dc.BWD_FILTER_NOALLOC_MAX_BYTES
        ws = torch.empty(need, dtype=torch.uint8, device="cuda")
        start = torch.randn((L.K, L.C, L.R, L.S), device="cuda")
        ref = start.clone()
        got = start.clone()
        dc.conv_bwd_filter(p, tile, xp, dyp, ref, acc, ws)
        dc.conv_bwd_filter_noalloc(p, tile, xp, dyp, got, acc)
        torch.cuda.synchronize()
        assert bool(torch.isfinite(got).all())
        assert torch.equal(_bits(got), _bits(ref)), L.name
        # a second call on the same inputs reuses the array: same bits again
        again = start.clone()
        dc.conv_bwd_filter_noalloc(p, tile, xp, dyp, again, acc)
        torch.cuda.synchronize()
        assert torch.equal(_bits(again), _bits(ref)), L.name
        del xp, dyp, ws
