"""Interior / boundary split of the forward and input-gradient passes
(Sec. IV-A: the halo exchange overlaps the interior computation).

A tile's outputs that read no margin are computed first (INTERIOR), the frame
of outputs that do afterwards (BOUNDARY).  The composition must equal the
undecomposed oracle element by element (bit for bit on integer inputs), with
the margins still NaN while the interior runs; BOUNDARY must write nothing
outside the frame; and the overlapped schedule (interior on one stream while
the halo is unpacked on another) must give the same bits as the serial one.
"""
import numpy as np
import pytest
import torch

import harness as H
import oracle as orc
import paper_1903_06681_amd as dc
import workloads as wl
from workloads import Layer

pytestmark = pytest.mark.gpu

X, DY, ALL = dc.DC_X, dc.DC_DY, dc.DC_ALL_TILES
INT, BND = dc.DC_REGION_INTERIOR, dc.DC_REGION_BOUNDARY
TOL = {"f32": 1e-5, "bf16": 2e-2}


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()


LAYERS = {
    # rolling-row kernel (3x3, 64 channels, 128-column strips)
    "roll": Layer("roll", 1, 64, 64, 256, 256, 3, 3, 1, 1, 2, 2, 1, "bf16", "uniform", 201),
    # register-weight strip kernel, partial strips, 3x3 grid
    "wreg": wl.small("c5a", N=2, H=96, W=96, P=3, Q=3),
    # 5x5: frame two wide; rolling-row 5x5 instantiation
    "roll5": Layer("roll5", 1, 32, 32, 256, 256, 5, 5, 1, 2, 1, 2, 2, "bf16", "uniform", 202),
    # fp32 register kernel (mesh layer), ragged tiles of the chunked kernel
    "f32": wl.small("c4", H=96, W=80, P=3, Q=2),
    "odd": Layer("odd", 2, 5, 7, 26, 39, 3, 3, 1, 1, 2, 3, 2, "bf16", "uniform", 203),
    "odd32": Layer("odd32", 2, 5, 7, 26, 39, 3, 3, 1, 1, 2, 3, 2, "f32", "uniform", 204),
    # frame kernel: two channel chunks (96 = 64 + 32 of 64), 40 output
    # channels (a partial 32-channel block); 7x7 (bands three wide, 98 groups)
    "wide": Layer("wide", 2, 96, 40, 64, 80, 3, 3, 1, 1, 2, 2, 1, "bf16", "uniform", 205),
    "k7": Layer("k7", 1, 16, 24, 48, 72, 7, 7, 1, 3, 2, 2, 3, "bf16", "uniform", 206),
    # frame kernel: 24 channels (a 3-group chunk: the runtime instantiation);
    # 128 -> 64 channels (whole chunks, weights copied raw, two chunks)
    "c24": Layer("c24", 2, 24, 32, 40, 56, 3, 3, 1, 1, 2, 2, 1, "bf16", "uniform", 207),
    "deep": Layer("deep", 2, 128, 64, 48, 64, 3, 3, 1, 1, 2, 2, 1, "bf16", "uniform", 208),
    # fp32 frame kernel: 5x5 (the runtime instantiation), 40 channels in
    # chunks of 16 (the last one partial), 24 output channels
    "f32k5": Layer("f32k5", 1, 40, 24, 40, 48, 5, 5, 1, 2, 2, 2, 2, "f32", "uniform", 209),
    # 5x5 tiles with three-wide bands: the frame is the whole tile (bottom
    # rows clamped, no side segments)
    "tiny7": Layer("tiny7", 2, 8, 8, 10, 10, 7, 7, 1, 3, 2, 2, 3, "bf16", "uniform", 210),
    "tiny7f": Layer("tiny7f", 2, 8, 8, 10, 10, 7, 7, 1, 3, 2, 2, 3, "f32", "uniform", 211),
    # 1x1 filter: no band, an empty frame (the boundary call launches nothing)
    "k1": Layer("k1", 2, 16, 24, 32, 48, 1, 1, 1, 0, 2, 2, 1, "bf16", "uniform", 212),
    "k1f": Layer("k1f", 2, 16, 24, 32, 48, 1, 1, 1, 0, 2, 2, 1, "f32", "uniform", 213),
}


def _bits(t):
    return t.view(torch.int16 if t.element_size() == 2 else torch.int32)


def _rel(g, r):
    g, r = np.asarray(g, np.float64), np.asarray(r, np.float64)
    assert np.all(np.isfinite(g))
    return float(np.max(np.abs(g - r)) / max(np.max(np.abs(r)), 1e-30))


def _frame_mask(th, tw, b):
    m = np.zeros((th, tw), bool)
    m[:b[0], :] = True
    m[th - b[1]:, :] = True
    m[:, :b[2]] = True
    m[:, tw - b[3]:] = True
    return m


def _setup(L, dist=None):
    p = dc.Problem.of(L)
    nt = L.P * L.Q
    x, w, dy = (wl.draw(L, t, dist=dist) for t in ("x", "w", "dy"))
    xt = H.alloc_tiles(p, X, nt, L.dtype)      # margins NaN
    dyt = H.alloc_tiles(p, DY, nt, L.dtype)
    H.scatter_interiors(xt, H.to_device(x, L.dtype), p, X)
    H.scatter_interiors(dyt, H.to_device(dy, L.dtype), p, DY)
    return p, x, w, dy, xt, dyt, H.to_device(w, L.dtype)


def _split(L, p, xt, dyt, wd, sa, sb=None):
    """interior passes (margins not yet filled), halo exchange (all tiles), boundary passes;
    with sb the exchange runs on stream sb beside the interior on sa"""
    nt = L.P * L.Q
    y = torch.full((nt, L.N, L.K, L.Hot, L.Wot), float("nan"), device="cuda")
    dx = torch.full((nt, L.N, L.C, L.Ht, L.Wt), float("nan"), device="cuda")
    sx = torch.empty((nt, dc.halo_elems(p, X)), dtype=xt.dtype, device="cuda")
    sy = torch.empty((nt, dc.halo_elems(p, DY)), dtype=dyt.dtype, device="cuda")
    ex = sb or sa
    if sb is not None:
        sb.wait_stream(sa)
    dc.conv_fwd_region(p, ALL, INT, xt, wd, y, sa)
    dc.conv_bwd_data_region(p, ALL, INT, dyt, wd, dx, sa)
    dc.halo_pack(p, ALL, X, xt, sx, ex)
    dc.halo_unpack(p, ALL, X, sx, xt, ex)
    dc.halo_pack(p, ALL, DY, dyt, sy, ex)
    dc.halo_unpack(p, ALL, DY, sy, dyt, ex)
    if sb is not None:
        sa.wait_stream(sb)
    dc.conv_fwd_region(p, ALL, BND, xt, wd, y, sa)
    dc.conv_bwd_data_region(p, ALL, BND, dyt, wd, dx, sa)
    torch.cuda.synchronize()
    return y, dx


@pytest.mark.parametrize("name", list(LAYERS))
@pytest.mark.parametrize("dist", [None, "int"])
def test_interior_then_boundary_matches_undecomposed_oracle(name, dist):
    L = LAYERS[name]
    print(f"[split] {name} {dist or L.dist}", flush=True)
    p, x, w, dy, xt, dyt, wd = _setup(L, dist)
    sa = torch.cuda.current_stream()
    y, dx = _split(L, p, xt, dyt, wd, sa)
    yg = H.gather_outputs(y, p, "y").cpu().numpy()
    dxg = H.gather_outputs(dx, p, "dx").cpu().numpy()
    yr = orc.round_f32(orc.conv_fwd(x, w, L.stride, L.pad))
    dxr = orc.round_f32(orc.conv_bwd_data(dy, w, L.H, L.W, L.stride, L.pad))
    if dist == "int":
        assert np.array_equal(yg, yr) and np.array_equal(dxg, dxr)
    else:
        assert _rel(yg, yr) <= TOL[L.dtype]
        assert _rel(dxg, dxr) <= TOL[L.dtype]


@pytest.mark.parametrize("name", list(LAYERS))
def test_boundary_writes_only_the_frame(name):
    L = LAYERS[name]
    p, x, w, dy, xt, dyt, wd = _setup(L)
    H.fill_halos_all_tiles(p, X, xt, L.dtype)
    H.fill_halos_all_tiles(p, DY, dyt, L.dtype)
    nt = L.P * L.Q
    sentinel = 1234.5
    y = torch.full((nt, L.N, L.K, L.Hot, L.Wot), sentinel, device="cuda")
    dx = torch.full((nt, L.N, L.C, L.Ht, L.Wt), sentinel, device="cuda")
    dc.conv_fwd_region(p, ALL, BND, xt, wd, y)
    dc.conv_bwd_data_region(p, ALL, BND, dyt, wd, dx)
    torch.cuda.synchronize()
    for out, bw, th, tw in ((y, dc.halo_bands(p, X), L.Hot, L.Wot), (dx, dc.halo_bands(p, DY), L.Ht, L.Wt)):
        fm = torch.from_numpy(_frame_mask(th, tw, bw)).cuda()
        untouched = (out == sentinel)
        assert bool(untouched[..., ~fm].all()), "wrote outside the frame"
        assert not bool(untouched[..., fm].any()), "left part of the frame"


@pytest.mark.parametrize("name", ["roll", "wreg", "f32"])
def test_overlapped_split_schedule_equals_serial(name):
    L = LAYERS[name]
    p, x, w, dy, xt, dyt, wd = _setup(L)
    sa = torch.cuda.current_stream()
    xt2, dyt2 = xt.clone(), dyt.clone()
    y1, dx1 = _split(L, p, xt, dyt, wd, sa)
    sb = torch.cuda.Stream()   # default priority
    for _ in range(3):
        xt3, dyt3 = xt2.clone(), dyt2.clone()   # margins NaN again
        y2, dx2 = _split(L, p, xt3, dyt3, wd, sa, sb)
        assert torch.equal(_bits(y1), _bits(y2)) and torch.equal(_bits(dx1), _bits(dx2))
