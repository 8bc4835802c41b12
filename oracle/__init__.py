"""CPU oracle for one GPU's share of a spatially decomposed convolution layer.

TEST INFRASTRUCTURE.  Only the test suite, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  The product
library never does, and this package imports nothing from it: the two share
no kernels, headers, helpers, tables or geometry code.

What it computes (Dryden et al., arXiv 1903.06681):

* ``conv_fwd`` / ``conv_bwd_data`` / ``conv_bwd_filter`` -- Eqs. (1), (3), (2)
  of Sec. II-A, generalised to stride and padding, as direct loops in
  ``oracle.c`` with fp64 accumulation (see the header there).  Results are
  fp64; ``round_f32`` rounds them once, to nearest-even, as the reference value.
* ``tile_window`` / ``halo_pack`` / ``halo_unpack`` -- the halo of Sec. III-A:
  a processor owning the blocked index ranges [q_H, r_H] x [q_W, r_W] needs
  the elements of ({q_H-O..q_H-1} u I_H u {r_H+1..r_H+O}) x (same in W) that it
  does not own, corners included; out-of-domain elements are the zero padding.
  These are pure index-set computations in numpy.
* ``tiled_*`` -- the decomposed computation of Sec. III-A: every tile runs the
  plain convolution on its own block plus halo, and the weight-gradient
  partials are summed over tiles (the allreduce) in row-major tile order.

Parity notes: the convolution functions are pinned by the tests in
``tests/test_oracle.py`` (hand cases, a library convolution, finite
differences, the adjoint identity, exact integer arithmetic and the
decomposition invariant); the sampled-point functions by bit-identity with
the whole-tensor ones at random, first and last flat indices; the halo
functions by brute-force index checks.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

_I64 = ctypes.c_int64
_PF = ctypes.POINTER(ctypes.c_float)
_PD = ctypes.POINTER(ctypes.c_double)
_PI = ctypes.POINTER(ctypes.c_int64)


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _b
        _b.build()
    lib = ctypes.CDLL(_LIB_PATH)
    dims = [_I64] * 11
    for name in ("oracle_conv_fwd", "oracle_conv_bwd_data", "oracle_conv_bwd_filter"):
        getattr(lib, name).argtypes = dims + [_PF, _PF, _PD]
        getattr(lib, name).restype = None
    for name in ("oracle_conv_fwd_points", "oracle_conv_bwd_data_points",
                 "oracle_conv_bwd_filter_points"):
        getattr(lib, name).argtypes = dims + [_PF, _PF, _PI, _I64, _PD]
        getattr(lib, name).restype = None
    lib.oracle_num_threads.argtypes = []
    lib.oracle_num_threads.restype = ctypes.c_int
    lib.oracle_set_num_threads.argtypes = [ctypes.c_int]
    lib.oracle_set_num_threads.restype = None
    _lib = lib
    return lib


def num_threads() -> int:
    """OpenMP threads the oracle's loops run on."""
    return int(_load().oracle_num_threads())


def set_num_threads(n: int) -> None:
    """Run the oracle's loops on n threads from now on."""
    _load().oracle_set_num_threads(int(n))


def _f32(a) -> np.ndarray:
    a = np.ascontiguousarray(a)
    if a.dtype != np.float32:
        raise TypeError("oracle inputs are fp32 arrays (bf16 values widened exactly)")
    return a


def _fp(a):
    return a.ctypes.data_as(_PF)


def out_size(n_in: int, r: int, stride: int, pad: int) -> int:
    """Output extent of a strided, padded convolution along one axis."""
    return (n_in + 2 * pad - r) // stride + 1


# --------------------------------------------------------------------------
# Convolutions, Eqs. (1)-(3)
# --------------------------------------------------------------------------

def conv_fwd(x, w, stride: int = 1, pad: int = 0) -> np.ndarray:
    """y = Eq. (1): x [N,C,Hi,Wi], w [K,C,R,S] -> y [N,K,Ho,Wo] in fp64."""
    x, w = _f32(x), _f32(w)
    N, C, Hi, Wi = x.shape
    K, C2, R, S = w.shape
    assert C2 == C
    Ho, Wo = out_size(Hi, R, stride, pad), out_size(Wi, S, stride, pad)
    y = np.empty((N, K, Ho, Wo), np.float64)
    _load().oracle_conv_fwd(N, C, K, Hi, Wi, Ho, Wo, R, S, stride, pad,
                            _fp(x), _fp(w), y.ctypes.data_as(_PD))
    return y


def conv_bwd_data(dy, w, Hi: int, Wi: int, stride: int = 1, pad: int = 0) -> np.ndarray:
    """dx = Eq. (3): dy [N,K,Ho,Wo], w [K,C,R,S] -> dx [N,C,Hi,Wi] in fp64."""
    dy, w = _f32(dy), _f32(w)
    N, K, Ho, Wo = dy.shape
    K2, C, R, S = w.shape
    assert K2 == K
    dx = np.empty((N, C, Hi, Wi), np.float64)
    _load().oracle_conv_bwd_data(N, C, K, Hi, Wi, Ho, Wo, R, S, stride, pad,
                                 _fp(dy), _fp(w), dx.ctypes.data_as(_PD))
    return dx


def conv_bwd_filter(x, dy, R: int, S: int, stride: int = 1, pad: int = 0) -> np.ndarray:
    """dw = Eq. (2): x [N,C,Hi,Wi], dy [N,K,Ho,Wo] -> dw [K,C,R,S] in fp64."""
    x, dy = _f32(x), _f32(dy)
    N, C, Hi, Wi = x.shape
    N2, K, Ho, Wo = dy.shape
    assert N2 == N
    dw = np.empty((K, C, R, S), np.float64)
    _load().oracle_conv_bwd_filter(N, C, K, Hi, Wi, Ho, Wo, R, S, stride, pad,
                                   _fp(x), _fp(dy), dw.ctypes.data_as(_PD))
    return dw


def _points(fn, dims, a, b, idx):
    idx = np.ascontiguousarray(idx, dtype=np.int64)
    out = np.empty(idx.shape[0], np.float64)
    fn(*dims, _fp(a), _fp(b), idx.ctypes.data_as(_PI), idx.shape[0],
       out.ctypes.data_as(_PD))
    return out


def conv_fwd_points(x, w, stride, pad, flat_idx) -> np.ndarray:
    """Eq. (1) at the given flat indices of y only (fp64)."""
    x, w = _f32(x), _f32(w)
    N, C, Hi, Wi = x.shape
    K, _, R, S = w.shape
    Ho, Wo = out_size(Hi, R, stride, pad), out_size(Wi, S, stride, pad)
    return _points(_load().oracle_conv_fwd_points,
                   (N, C, K, Hi, Wi, Ho, Wo, R, S, stride, pad), x, w, flat_idx)


def conv_bwd_data_points(dy, w, Hi, Wi, stride, pad, flat_idx) -> np.ndarray:
    """Eq. (3) at the given flat indices of dx only (fp64)."""
    dy, w = _f32(dy), _f32(w)
    N, K, Ho, Wo = dy.shape
    _, C, R, S = w.shape
    return _points(_load().oracle_conv_bwd_data_points,
                   (N, C, K, Hi, Wi, Ho, Wo, R, S, stride, pad), dy, w, flat_idx)


def conv_bwd_filter_points(x, dy, R, S, stride, pad, flat_idx) -> np.ndarray:
    """Eq. (2) at the given flat indices of dw only (fp64)."""
    x, dy = _f32(x), _f32(dy)
    N, C, Hi, Wi = x.shape
    _, K, Ho, Wo = dy.shape
    return _points(_load().oracle_conv_bwd_filter_points,
                   (N, C, K, Hi, Wi, Ho, Wo, R, S, stride, pad), x, dy, flat_idx)


def round_f32(a: np.ndarray) -> np.ndarray:
    """Round fp64 results once to fp32, to nearest-even."""
    return np.asarray(a, np.float64).astype(np.float32)


# --------------------------------------------------------------------------
# Blocked spatial distribution and the halo set (Sec. III-A)
# --------------------------------------------------------------------------

# The packed halo buffer layout of the library interface: eight regions in
# this order, each [N][channels][rows][cols], at offsets fixed by the nominal
# region sizes.  (A format both sides must agree on, restated here.)
DIRECTIONS = ("N", "S", "W", "E", "NW", "NE", "SW", "SE")
STEP = {"N": (-1, 0), "S": (1, 0), "W": (0, -1), "E": (0, 1),
        "NW": (-1, -1), "NE": (-1, 1), "SW": (1, -1), "SE": (1, 1)}
OPPOSITE = {"N": "S", "S": "N", "W": "E", "E": "W",
            "NW": "SE", "NE": "SW", "SW": "NE", "SE": "NW"}


def owned_ranges(H, W, P, Q, ti, tj):
    """Blocked index ranges [q_H, r_H] x [q_W, r_W] (inclusive) of tile (ti, tj)."""
    Ht, Wt = H // P, W // Q
    return (ti * Ht, ti * Ht + Ht - 1), (tj * Wt, tj * Wt + Wt - 1)


def _bands(h, bw):
    """Band widths (above, below, left, right); None means h on every side."""
    return (h, h, h, h) if bw is None else tuple(int(v) for v in bw)


def window_ranges(H, W, P, Q, ti, tj, h, bw=None):
    """Owned block widened by its halo bands (global indices, inclusive): h on
    every side, or bw = (above, below, left, right)."""
    a, b, l, r = _bands(h, bw)
    (qh, rh), (qw, rw) = owned_ranges(H, W, P, Q, ti, tj)
    return (qh - a, rh + b), (qw - l, rw + r)


def tile_window(g: np.ndarray, P, Q, ti, tj, h, bw=None) -> np.ndarray:
    """Owned block of tile (ti,tj) plus an h-wide margin, read from the global
    tensor g [N,C,H,W]; margin cells outside the domain are zero, and so are
    cells outside the halo bands bw = (above, below, left, right) when given
    (the part of the margin no pass reads)."""
    N, C, H, W = g.shape
    (a0, a1), (b0, b1) = window_ranges(H, W, P, Q, ti, tj, h)
    (qa, qb), (ql, qr) = window_ranges(H, W, P, Q, ti, tj, h, bw)
    out = np.zeros((N, C, a1 - a0 + 1, b1 - b0 + 1), g.dtype)
    for i in range(max(a0, qa), min(a1, qb) + 1):
        if 0 <= i < H:
            lo, hi = max(b0, ql, 0), min(b1, qr, W - 1)
            if lo <= hi:
                out[:, :, i - a0, lo - b0:hi - b0 + 1] = g[:, :, i, lo:hi + 1]
    return out


def halo_mask(Ht, Wt, h) -> np.ndarray:
    """True on the halo part of a (Ht+2h) x (Wt+2h) window, False on the owned block."""
    m = np.ones((Ht + 2 * h, Wt + 2 * h), bool)
    m[h:h + Ht, h:h + Wt] = False
    return m


def _intersect(a, b):
    lo, hi = max(a[0], b[0]), min(a[1], b[1])
    return (lo, hi) if lo <= hi else None


def region_shapes(Ht, Wt, h, bw=None, send=False):
    """(rows, cols) of each packed region.  A receive region d is the band of
    margin d; a send region d is what the neighbour in direction d receives,
    the band of ITS margin opposite to d."""
    a, b, l, r = _bands(h, bw)
    rows = {-1: a, 0: Ht, 1: b}
    cols = {-1: l, 0: Wt, 1: r}
    out = {}
    for d in DIRECTIONS:
        di, dj = STEP[OPPOSITE[d]] if send else STEP[d]
        out[d] = (rows[di], cols[dj])
    return out


def region_offsets(N, Cc, Ht, Wt, h, bw=None, send=False):
    """Element offset of each region in one tile's packed buffer, and the total."""
    offs, o = {}, 0
    for d, (r, c) in region_shapes(Ht, Wt, h, bw, send).items():
        offs[d] = o
        o += N * Cc * r * c
    return offs, o


def neighbour(P, Q, ti, tj, d):
    di, dj = STEP[d]
    ni, nj = ti + di, tj + dj
    return (ni, nj) if (0 <= ni < P and 0 <= nj < Q) else None


def pack_region_ranges(H, W, P, Q, ti, tj, h, d, bw=None):
    """Global index ranges that tile (ti,tj) sends toward direction d: the part
    of its owned block lying in the neighbour's halo window.  None if no
    neighbour exists (nothing is sent)."""
    nb = neighbour(P, Q, ti, tj, d)
    if nb is None:
        return None
    own_h, own_w = owned_ranges(H, W, P, Q, ti, tj)
    win_h, win_w = window_ranges(H, W, P, Q, nb[0], nb[1], h, bw)
    rh, rw = _intersect(own_h, win_h), _intersect(own_w, win_w)
    if rh is None or rw is None:
        return (0, -1), (0, -1)   # an empty band
    return rh, rw


def halo_pack(g: np.ndarray, P, Q, ti, tj, h, send: np.ndarray, bw=None) -> np.ndarray:
    """Fill tile (ti,tj)'s packed send buffer from the global tensor g.
    Regions without a neighbour are left as they were."""
    N, C, H, W = g.shape
    Ht, Wt = H // P, W // Q
    offs, total = region_offsets(N, C, Ht, Wt, h, bw, send=True)
    shapes = region_shapes(Ht, Wt, h, bw, send=True)
    assert send.shape == (total,)
    for d in DIRECTIONS:
        rng = pack_region_ranges(H, W, P, Q, ti, tj, h, d, bw)
        if rng is None:
            continue
        (a0, a1), (b0, b1) = rng
        blk = g[:, :, a0:a1 + 1, b0:b1 + 1]
        if 0 in shapes[d]:
            continue
        assert blk.shape[2:] == shapes[d]
        send[offs[d]:offs[d] + blk.size] = blk.reshape(-1)
    return send


def halo_unpack(recv: np.ndarray, N, C, H, W, P, Q, ti, tj, h, window: np.ndarray, bw=None) -> np.ndarray:
    """Write the halo part of tile (ti,tj)'s window [N,C,Ht+2h,Wt+2h].

    ``recv`` is the tile's packed receive buffer: its region d holds what the
    neighbour in direction d sent (see ``gather_recv``).  The band of margin d
    takes region d where the neighbour exists; every other margin cell (no
    neighbour: the domain's zero padding; outside the bands: never read) is
    zero.  The owned block is untouched."""
    Ht, Wt = H // P, W // Q
    a, b, l, r = _bands(h, bw)
    offs, _ = region_offsets(N, C, Ht, Wt, h, bw)
    window[:, :, :h, :] = 0
    window[:, :, h + Ht:, :] = 0
    window[:, :, :, :h] = 0
    window[:, :, :, h + Wt:] = 0
    for d in DIRECTIONS:
        di, dj = STEP[d]
        # the band of margin d, in window coordinates (inclusive)
        rows = {-1: (h - a, h - 1), 0: (h, h + Ht - 1), 1: (h + Ht, h + Ht + b - 1)}[di]
        cols = {-1: (h - l, h - 1), 0: (h, h + Wt - 1), 1: (h + Wt, h + Wt + r - 1)}[dj]
        nr, nc = rows[1] - rows[0] + 1, cols[1] - cols[0] + 1
        if nr <= 0 or nc <= 0 or neighbour(P, Q, ti, tj, d) is None:
            continue
        blk = recv[offs[d]:offs[d] + N * C * nr * nc].reshape(N, C, nr, nc)
        window[:, :, rows[0]:rows[1] + 1, cols[0]:cols[1] + 1] = blk
    return window


def gather_recv(sends: dict, N, C, H, W, P, Q, ti, tj, h, bw=None) -> np.ndarray:
    """Assemble tile (ti,tj)'s receive buffer: region d := neighbour d's send
    region OPPOSITE[d].  Regions without a neighbour are zero."""
    Ht, Wt = H // P, W // Q
    offs, total = region_offsets(N, C, Ht, Wt, h, bw)
    soffs, _ = region_offsets(N, C, Ht, Wt, h, bw, send=True)
    shapes = region_shapes(Ht, Wt, h, bw)
    recv = np.zeros(total, next(iter(sends.values())).dtype)
    for d in DIRECTIONS:
        nb = neighbour(P, Q, ti, tj, d)
        if nb is None:
            continue
        o = OPPOSITE[d]
        n = N * C * shapes[d][0] * shapes[d][1]
        recv[offs[d]:offs[d] + n] = sends[nb][soffs[o]:soffs[o] + n]
    return recv


# --------------------------------------------------------------------------
# Needed halo widths, by brute force over the index sets the sums touch
# --------------------------------------------------------------------------

def needed_halo_x(Hi, R, stride, pad, Ho, Ht, Hot, t0_out, t0_in):
    """Rows of x outside [t0_in, t0_in+Ht) that Eq. (1) reads for output rows
    [t0_out, t0_out+Hot): returns (below, above) counts."""
    lo = hi = 0
    for p in range(t0_out, t0_out + Hot):
        for r in range(R):
            i = p * stride - pad + r
            lo = max(lo, t0_in - i)
            hi = max(hi, i - (t0_in + Ht - 1))
    return lo, hi


def needed_halo_dy(Ho, R, stride, pad, Ht, Hot, t0_in, t0_out):
    """Rows of dy outside [t0_out, t0_out+Hot) that Eq. (3) reads for input
    rows [t0_in, t0_in+Ht): returns (below, above) counts."""
    lo = hi = 0
    for i in range(t0_in, t0_in + Ht):
        for r in range(R):
            t = i + pad - r
            if t % stride:
                continue
            p = t // stride
            lo = max(lo, t0_out - p)
            hi = max(hi, p - (t0_out + Hot - 1))
    return lo, hi


def halo_bands(which, H, W, R, S, stride, pad, P, Q):
    """Band widths (above, below, left, right) a tile's passes read beyond it:
    x for Eq. (1)/(2), dy for Eq. (3), by brute force over the index sets of
    the first tile (every tile of an aligned grid reads the same margins)."""
    Ho, Wo = out_size(H, R, stride, pad), out_size(W, S, stride, pad)
    Ht, Wt, Hot, Wot = H // P, W // Q, Ho // P, Wo // Q
    if which == "x":
        rows = needed_halo_x(H, R, stride, pad, Ho, Ht, Hot, 0, 0)
        cols = needed_halo_x(W, S, stride, pad, Wo, Wt, Wot, 0, 0)
    else:
        rows = needed_halo_dy(Ho, R, stride, pad, Ht, Hot, 0, 0)
        cols = needed_halo_dy(Wo, S, stride, pad, Wt, Wot, 0, 0)
    return rows[0], rows[1], cols[0], cols[1]


# --------------------------------------------------------------------------
# Decomposed (tiled) computation, Sec. III-A
# --------------------------------------------------------------------------

def tiled_conv(x, w, dy, P, Q, h, pad, stride=1, bands=False):
    """Decomposed forward, backward-data and backward-filter over a P x Q grid
    of blocked tiles with halo width h >= needed (Sec. III-A).  With stride s
    an input tile of Ht x Wt owns the Ht/s x Wt/s output block whose taps start
    in it.  Every tile works on its own window (owned block plus h on every
    side, zeros outside the domain):
      y:  Eq. (1) over the window rows from h - pad on, pad 0;
      dx: Eq. (3) over the whole dy window, whose row 0 sits h output rows
          above the tile, so the taps are shifted by h*s (pad + h*s);
      dw: Eq. (2) over the dy interior and the same x rows as y.
    y and dx are stitched; the dw partials are summed in fp64 in row-major
    tile order.  With bands=True each window holds only the halo bands of
    ``halo_bands`` (zeros in the rest of the margin).  Returns (y, dx, dw) in
    fp64."""
    N, C, H, W = x.shape
    K, _, R, S = w.shape
    Ht, Wt = H // P, W // Q
    Hot, Wot = Ht // stride, Wt // stride
    nr, ns = (Hot - 1) * stride + R, (Wot - 1) * stride + S   # x rows/cols one tile reads
    y = np.zeros((N, K, Hot * P, Wot * Q))
    dx = np.zeros((N, C, H, W))
    dw = np.zeros((K, C, R, S))
    for ti in range(P):
        for tj in range(Q):
            bx = halo_bands("x", H, W, R, S, stride, pad, P, Q) if bands else None
            by = halo_bands("dy", H, W, R, S, stride, pad, P, Q) if bands else None
            xw = tile_window(x, P, Q, ti, tj, h, bx)
            dyw = tile_window(dy, P, Q, ti, tj, h, by)    # dy tiles are Hot x Wot, same grid
            xs = np.ascontiguousarray(xw[:, :, h - pad:h - pad + nr, h - pad:h - pad + ns])
            yt = conv_fwd(xs, w, stride, 0)
            dxt = conv_bwd_data(np.ascontiguousarray(dyw), w, Ht, Wt, stride, pad + h * stride)
            dyo = np.ascontiguousarray(dyw[:, :, h:h + Hot, h:h + Wot])
            dwt = conv_bwd_filter(xs, dyo, R, S, stride, 0)
            y[:, :, ti * Hot:(ti + 1) * Hot, tj * Wot:(tj + 1) * Wot] = yt
            dx[:, :, ti * Ht:(ti + 1) * Ht, tj * Wt:(tj + 1) * Wt] = dxt
            dw += dwt
    return y, dx, dw
