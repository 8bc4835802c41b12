"""Pins for the CPU oracle (no GPU).

Each test checks the oracle against something other than itself: values fixed
by hand from Eq. (1), a library convolution, finite differences of the
forward pass, the adjoint identity that ties Eqs. (1)-(3) together, exact
integer arithmetic, and the paper's claim that the decomposed computation
reproduces the undecomposed one (Sec. III).  A plausible mistake in the
oracle -- a flipped filter, a dropped tap, a wrong stride or padding offset,
a transposed weight index -- fails at least one of them.
"""
import itertools

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle as orc


def _rand(rng, shape, kind="real"):
    if kind == "int":
        return rng.integers(-2, 3, size=shape).astype(np.float32)
    return rng.uniform(-1, 1, size=shape).astype(np.float32)


# ---------------------------------------------------------------- hand cases

@pytest.mark.parametrize("C", [1, 3])
def test_all_ones_counts_in_range_taps(C):
    """Eq. (1) with x = w = 1, 3x3, 'same' padding: y = C x (#taps inside the
    image): 4C at corners, 6C on edges, 9C inside."""
    x = np.ones((1, C, 4, 5), np.float32)
    w = np.ones((2, C, 3, 3), np.float32)
    y = orc.conv_fwd(x, w, 1, 1)
    expect = np.full((4, 5), 9.0 * C)
    expect[0, :] = expect[-1, :] = 6.0 * C
    expect[:, 0] = expect[:, -1] = 6.0 * C
    for i, j in [(0, 0), (0, -1), (-1, 0), (-1, -1)]:
        expect[i, j] = 4.0 * C
    assert np.array_equal(y[0, 0], expect) and np.array_equal(y[0, 1], expect)


@pytest.mark.parametrize("R,pad", [(3, 1), (5, 2)])
def test_delta_filter_shifts_without_flip(R, pad):
    """A filter that is 1 at (r,s) and 0 elsewhere gives y[p,q] = x[p+r-pad, q+s-pad]
    (zero outside): cross-correlation, no flip."""
    rng = np.random.default_rng(7)
    x = _rand(rng, (1, 1, 6, 7))
    for r, s in itertools.product(range(R), range(R)):
        w = np.zeros((1, 1, R, R), np.float32)
        w[0, 0, r, s] = 1
        y = orc.conv_fwd(x, w, 1, pad)
        expect = np.zeros((6, 7))
        for p in range(6):
            for q in range(7):
                i, j = p + r - pad, q + s - pad
                if 0 <= i < 6 and 0 <= j < 7:
                    expect[p, q] = x[0, 0, i, j]
        assert np.array_equal(y[0, 0], expect), (r, s)


def test_one_by_one_is_a_matrix_product():
    """A 1x1 conv is y[n,:,p,q] = W x[n,:,p,q] (textbook matrix product)."""
    rng = np.random.default_rng(3)
    x = _rand(rng, (2, 5, 4, 3))
    w = _rand(rng, (6, 5, 1, 1))
    y = orc.conv_fwd(x, w, 1, 0)
    ref = np.einsum("kc,nchw->nkhw", w[:, :, 0, 0].astype(np.float64), x.astype(np.float64))
    np.testing.assert_allclose(y, ref, rtol=1e-13, atol=1e-13)


def test_stride_two_is_subsampled_stride_one():
    """A stride-2 conv equals the stride-1 conv at the same padding, sampled
    at even output positions."""
    rng = np.random.default_rng(11)
    x = _rand(rng, (1, 2, 9, 8))
    w = _rand(rng, (3, 2, 3, 3))
    y1 = orc.conv_fwd(x, w, 1, 1)
    y2 = orc.conv_fwd(x, w, 2, 1)
    assert np.array_equal(y2, y1[:, :, ::2, ::2])


# ------------------------------------------------------ library convolution

CASES = [
    # N, C, K, H, W, R, S, stride, pad
    (1, 1, 1, 5, 5, 3, 3, 1, 1),
    (2, 3, 4, 7, 6, 3, 3, 1, 1),
    (2, 3, 2, 9, 9, 5, 5, 1, 2),
    (1, 2, 3, 8, 8, 1, 1, 1, 0),
    (2, 3, 4, 11, 10, 7, 7, 2, 3),
    (1, 2, 2, 9, 7, 3, 3, 2, 1),
    (1, 2, 3, 6, 8, 3, 5, 1, 0),
    (1, 2, 2, 10, 9, 3, 3, 2, 0),
]


@pytest.mark.parametrize("case", CASES)
def test_matches_library_convolution_and_autograd(case):
    """fp64 torch conv2d and its autograd gradients compute Eqs. (1)-(3) on
    the CPU; the oracle must agree to fp64 rounding."""
    N, C, K, H, W, R, S, st, pad = case
    rng = np.random.default_rng(hash(case) % 2**32)
    x = _rand(rng, (N, C, H, W))
    w = _rand(rng, (K, C, R, S))
    y = orc.conv_fwd(x, w, st, pad)
    dy = _rand(rng, y.shape)
    xt = torch.from_numpy(x.astype(np.float64)).requires_grad_(True)
    wt = torch.from_numpy(w.astype(np.float64)).requires_grad_(True)
    yt = F.conv2d(xt, wt, stride=st, padding=pad)
    yt.backward(torch.from_numpy(dy.astype(np.float64)))
    np.testing.assert_allclose(y, yt.detach().numpy(), rtol=1e-12, atol=1e-12)
    dx = orc.conv_bwd_data(dy, w, H, W, st, pad)
    dw = orc.conv_bwd_filter(x, dy, R, S, st, pad)
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dw, wt.grad.numpy(), rtol=1e-12, atol=1e-11)


# --------------------------------------------------------- finite differences

FD_CASES = [(R, st, pad) for R in (1, 3, 5) for st in (1, 2) for pad in (0, 1, 2) if pad < R or R == 1 and pad == 0]


@pytest.mark.parametrize("R,st,pad", FD_CASES)
def test_gradients_by_central_differences(R, st, pad):
    """L = <y, dy> is linear in x and in w, so with integer-valued data and a
    unit step the central difference of the oracle's own forward pass is
    exact: it must reproduce Eqs. (2) and (3) element by element."""
    rng = np.random.default_rng(R * 100 + st * 10 + pad)
    N, C, K, H, W = 2, 2, 3, 6, 5
    x = _rand(rng, (N, C, H, W), "int")
    w = _rand(rng, (K, C, R, R), "int")
    Ho, Wo = orc.out_size(H, R, st, pad), orc.out_size(W, R, st, pad)
    if Ho <= 0 or Wo <= 0:
        pytest.skip("empty output")
    dy = _rand(rng, (N, K, Ho, Wo), "int")

    def L(xx, ww):
        return float(np.sum(orc.conv_fwd(xx, ww, st, pad) * dy))

    dx = orc.conv_bwd_data(dy, w, H, W, st, pad)
    dw = orc.conv_bwd_filter(x, dy, R, R, st, pad)
    for idx in np.ndindex(x.shape):
        xp, xm = x.copy(), x.copy()
        xp[idx] += 1
        xm[idx] -= 1
        assert (L(xp, w) - L(xm, w)) / 2 == dx[idx], idx
    for idx in np.ndindex(w.shape):
        wp, wm = w.copy(), w.copy()
        wp[idx] += 1
        wm[idx] -= 1
        assert (L(x, wp) - L(x, wm)) / 2 == dw[idx], idx


@pytest.mark.parametrize("case", CASES)
def test_adjoint_identity(case):
    """<conv(x,w), dy> = <x, dx> = <w, dw>: all three passes tie together."""
    N, C, K, H, W, R, S, st, pad = case
    rng = np.random.default_rng(5 + hash(case) % 1000)
    x = _rand(rng, (N, C, H, W))
    w = _rand(rng, (K, C, R, S))
    y = orc.conv_fwd(x, w, st, pad)
    dy = _rand(rng, y.shape)
    dx = orc.conv_bwd_data(dy, w, H, W, st, pad)
    dw = orc.conv_bwd_filter(x, dy, R, S, st, pad)
    a = np.sum(y * dy)
    b = np.sum(x.astype(np.float64) * dx)
    c = np.sum(w.astype(np.float64) * dw)
    scale = np.sum(np.abs(y * dy)) + 1.0
    assert abs(a - b) <= 1e-12 * scale and abs(a - c) <= 1e-12 * scale


def test_integer_inputs_are_exact():
    """Integer-valued inputs: every product and partial sum is an exact
    integer, so the oracle must equal an int64 evaluation of the sums."""
    rng = np.random.default_rng(19)
    N, C, K, H, W, R, st, pad = 2, 3, 2, 7, 6, 3, 1, 1
    x = _rand(rng, (N, C, H, W), "int")
    w = _rand(rng, (K, C, R, R), "int")
    y = orc.conv_fwd(x, w, st, pad)
    xi = np.pad(x.astype(np.int64), ((0, 0), (0, 0), (pad, pad), (pad, pad)))
    wi = w.astype(np.int64)
    yi = np.zeros((N, K, H, W), np.int64)
    for r in range(R):
        for s in range(R):
            yi += np.einsum("kc,nchw->nkhw", wi[:, :, r, s], xi[:, :, r:r + H, s:s + W])
    assert np.array_equal(y, yi.astype(np.float64))


# --------------------------------------------------------------- halo sets

def _brute_window(g, P, Q, ti, tj, h):
    N, C, H, W = g.shape
    Ht, Wt = H // P, W // Q
    out = np.empty((N, C, Ht + 2 * h, Wt + 2 * h), g.dtype)
    for a in range(Ht + 2 * h):
        for b in range(Wt + 2 * h):
            i, j = ti * Ht - h + a, tj * Wt - h + b
            out[:, :, a, b] = g[:, :, i, j] if (0 <= i < H and 0 <= j < W) else 0
    return out


@pytest.mark.parametrize("P,Q,h", [(1, 1, 1), (2, 2, 1), (2, 3, 2), (4, 4, 1), (3, 2, 3)])
def test_halo_round_trip_reproduces_padded_window(P, Q, h):
    """pack -> exchange -> unpack leaves every tile holding exactly its owned
    block plus the halo set of Sec. III-A (corners included), with zeros where
    the halo falls outside the domain; checked against per-element indexing."""
    rng = np.random.default_rng(P * 10 + Q + h)
    N, C, H, W = 2, 3, 6 * P, 6 * Q
    g = rng.standard_normal((N, C, H, W)).astype(np.float32)
    Ht, Wt = H // P, W // Q
    offs, total = orc.region_offsets(N, C, Ht, Wt, h)
    sends = {}
    for ti in range(P):
        for tj in range(Q):
            sends[(ti, tj)] = orc.halo_pack(g, P, Q, ti, tj, h, np.full(total, np.nan, np.float32))
    for ti in range(P):
        for tj in range(Q):
            win = np.full((N, C, Ht + 2 * h, Wt + 2 * h), np.nan, np.float32)
            win[:, :, h:h + Ht, h:h + Wt] = g[:, :, ti * Ht:(ti + 1) * Ht, tj * Wt:(tj + 1) * Wt]
            recv = orc.gather_recv(sends, N, C, H, W, P, Q, ti, tj, h)
            orc.halo_unpack(recv, N, C, H, W, P, Q, ti, tj, h, win)
            brute = _brute_window(g, P, Q, ti, tj, h)
            assert np.array_equal(win, brute)
            assert np.array_equal(orc.tile_window(g, P, Q, ti, tj, h), brute)


def _brute_band_window(g, P, Q, ti, tj, h, bw):
    """The padded window with zeros outside the bands (above, below, left, right)."""
    out = _brute_window(g, P, Q, ti, tj, h)
    N, C, H, W = g.shape
    Ht, Wt = H // P, W // Q
    a, b, l, r = bw
    for i in range(Ht + 2 * h):
        for j in range(Wt + 2 * h):
            if not (h - a <= i < h + Ht + b and h - l <= j < h + Wt + r):
                out[:, :, i, j] = 0
    return out


@pytest.mark.parametrize("P,Q,h,bw", [(2, 2, 3, (3, 2, 3, 2)), (3, 2, 2, (0, 1, 1, 0)),
                                      (2, 3, 2, (1, 2, 2, 1)), (4, 4, 1, (1, 0, 0, 1)),
                                      (2, 2, 2, (2, 2, 2, 2)), (1, 1, 2, (1, 1, 2, 0))])
def test_halo_round_trip_with_per_side_bands(P, Q, h, bw):
    """With band widths (above, below, left, right) narrower than the margin,
    pack -> exchange -> unpack fills each margin band from the neighbour,
    zeros the rest of the margin, and leaves the owned block alone; the send
    and receive buffers hold the same number of elements."""
    rng = np.random.default_rng(P * 10 + Q + h + sum(bw))
    N, C, H, W = 2, 3, 6 * P, 6 * Q
    g = rng.standard_normal((N, C, H, W)).astype(np.float32)
    Ht, Wt = H // P, W // Q
    _, total = orc.region_offsets(N, C, Ht, Wt, h, bw)
    _, stotal = orc.region_offsets(N, C, Ht, Wt, h, bw, send=True)
    assert total == stotal
    sends = {(ti, tj): orc.halo_pack(g, P, Q, ti, tj, h, np.full(total, np.nan, np.float32), bw)
             for ti in range(P) for tj in range(Q)}
    for ti in range(P):
        for tj in range(Q):
            win = np.full((N, C, Ht + 2 * h, Wt + 2 * h), np.nan, np.float32)
            win[:, :, h:h + Ht, h:h + Wt] = g[:, :, ti * Ht:(ti + 1) * Ht, tj * Wt:(tj + 1) * Wt]
            recv = orc.gather_recv(sends, N, C, H, W, P, Q, ti, tj, h, bw)
            orc.halo_unpack(recv, N, C, H, W, P, Q, ti, tj, h, win, bw)
            brute = _brute_band_window(g, P, Q, ti, tj, h, bw)
            assert np.array_equal(win, brute)
            assert np.array_equal(orc.tile_window(g, P, Q, ti, tj, h, bw), brute)


@pytest.mark.parametrize("R,stride,pad,x_bw,dy_bw", [
    (3, 1, 1, (1, 1, 1, 1), (1, 1, 1, 1)),
    (5, 1, 2, (2, 2, 2, 2), (2, 2, 2, 2)),
    (1, 1, 0, (0, 0, 0, 0), (0, 0, 0, 0)),
    (7, 2, 3, (3, 2, 3, 2), (1, 2, 1, 2)),   # ResNet conv1 on a grid
    (3, 2, 1, (1, 0, 1, 0), (0, 1, 0, 1)),   # stride-2 block entry: one-sided halos
])
def test_halo_bands_closed_forms(R, stride, pad, x_bw, dy_bw):
    """The bands the brute-force index sets give: x above = pad, below =
    max(0, R - pad - stride); dy above = floor((R-1-pad)/stride), below =
    floor((pad-1)/stride) + 1 (Sec. III-A: at stride > 1 a side may need no
    halo)."""
    H = W = 16 * stride
    assert orc.halo_bands("x", H, W, R, R, stride, pad, 4, 4) == x_bw
    assert orc.halo_bands("dy", H, W, R, R, stride, pad, 4, 4) == dy_bw
    assert x_bw[:2] == (pad, max(0, R - pad - stride))
    assert dy_bw[:2] == ((R - 1 - pad) // stride, (pad - 1) // stride + 1)


@pytest.mark.parametrize("P,Q,h,R,pad,stride,kind", [
    (2, 2, 3, 7, 3, 2, "int"), (4, 2, 3, 7, 3, 2, "real"), (2, 2, 1, 3, 1, 2, "int"),
    (2, 3, 2, 3, 1, 1, "int"), (2, 2, 2, 5, 2, 1, "real"),
])
def test_decomposed_with_bands_only_equals_undecomposed(P, Q, h, R, pad, stride, kind):
    """Windows that hold only the halo bands (zeros in the rest of the
    margin) still give the undecomposed result: the bands are all the passes
    read (y and dx bit for bit, dw bit for bit on integers)."""
    rng = np.random.default_rng(P * 100 + Q * 10 + h + R + stride)
    N, C, K = 2, 3, 4
    H, W = 4 * stride * P, 3 * stride * Q
    x = _rand(rng, (N, C, H, W), kind)
    w = _rand(rng, (K, C, R, R), kind)
    dy = _rand(rng, (N, K, H // stride, W // stride), kind)
    y0 = orc.round_f32(orc.conv_fwd(x, w, stride, pad))
    dx0 = orc.round_f32(orc.conv_bwd_data(dy, w, H, W, stride, pad))
    dw0 = orc.round_f32(orc.conv_bwd_filter(x, dy, R, R, stride, pad))
    y1, dx1, dw1 = (orc.round_f32(a) for a in orc.tiled_conv(x, w, dy, P, Q, h, pad, stride, bands=True))
    assert np.array_equal(y0, y1) and np.array_equal(dx0, dx1)
    if kind == "int":
        assert np.array_equal(dw0, dw1)
    else:
        assert np.all(np.abs(dw0.astype(np.float64) - dw1) <= np.abs(np.spacing(dw0)))


def test_halo_size_matches_message_terms():
    """An interior tile's halo holds 2*O*I_H + 2*O*I_W + 4*O^2 elements per
    (sample, channel): the east/west, north/south and corner terms of the
    forward-propagation cost FP_l (Sec. V-A)."""
    for Ht, Wt, h in [(5, 7, 1), (8, 8, 2), (4, 6, 3)]:
        assert orc.halo_mask(Ht, Wt, h).sum() == 2 * h * Ht + 2 * h * Wt + 4 * h * h
        _, total = orc.region_offsets(1, 1, Ht, Wt, h)
        assert total == 2 * h * Ht + 2 * h * Wt + 4 * h * h


def test_one_by_one_needs_no_halo():
    """K = 1 gives O = 0: no halo is needed (Sec. III-A)."""
    assert orc.needed_halo_x(8, 1, 1, 0, 8, 4, 4, 4, 4) == (0, 0)
    assert orc.needed_halo_dy(8, 1, 1, 0, 4, 4, 4, 4) == (0, 0)


def test_stride_two_may_need_no_halo_on_one_side():
    """3x3 stride 2 pad 1: the x halo is 1 below and 0 above (Sec. III-A: with
    stride > 1 some processors need no halo)."""
    # tile of 8 input rows at offset 8 -> 4 output rows at offset 4
    assert orc.needed_halo_x(16, 3, 2, 1, 8, 8, 4, 4, 8) == (1, 0)


# ------------------------------------------------- decomposition invariant

@pytest.mark.parametrize("P,Q,h,R,pad,kind", [
    (1, 1, 1, 3, 1, "real"), (2, 2, 1, 3, 1, "real"), (2, 3, 1, 3, 1, "real"),
    (4, 4, 1, 3, 1, "real"), (2, 2, 2, 5, 2, "real"), (2, 2, 2, 3, 1, "real"),
    (2, 2, 1, 3, 1, "int"), (4, 4, 2, 5, 2, "int"), (2, 2, 0, 1, 0, "real"),
])
def test_decomposed_equals_undecomposed(P, Q, h, R, pad, kind):
    """Sec. III: the spatially decomposed algorithm replicates the single-GPU
    convolution up to floating-point accumulation order.  y and dx use the
    same terms in the same order, so they match bit for bit; dw is summed per
    tile first, so it matches bit for bit on integer data and within one fp32
    ulp otherwise."""
    rng = np.random.default_rng(P * 1000 + Q * 100 + h * 10 + R)
    N, C, K = 2, 3, 4
    H, W = 4 * P, 5 * Q
    x = _rand(rng, (N, C, H, W), kind)
    w = _rand(rng, (K, C, R, R), kind)
    dy = _rand(rng, (N, K, H, W), kind)
    y0 = orc.round_f32(orc.conv_fwd(x, w, 1, pad))
    dx0 = orc.round_f32(orc.conv_bwd_data(dy, w, H, W, 1, pad))
    dw0 = orc.round_f32(orc.conv_bwd_filter(x, dy, R, R, 1, pad))
    y1, dx1, dw1 = (orc.round_f32(a) for a in orc.tiled_conv(x, w, dy, P, Q, h, pad))
    assert np.array_equal(y0, y1)
    assert np.array_equal(dx0, dx1)
    if kind == "int":
        assert np.array_equal(dw0, dw1)
    else:
        ulp = np.abs(np.spacing(dw0))
        assert np.all(np.abs(dw0.astype(np.float64) - dw1) <= ulp)



@pytest.mark.parametrize("P,Q,h,R,pad,stride,kind", [
    (2, 2, 1, 3, 1, 2, "real"), (2, 2, 1, 3, 1, 2, "int"), (4, 2, 3, 7, 3, 2, "real"),
    (2, 2, 3, 7, 3, 2, "int"), (2, 2, 0, 1, 0, 2, "real"), (2, 2, 1, 1, 0, 2, "real"),
    (3, 2, 2, 5, 2, 2, "real"), (2, 2, 1, 3, 1, 3, "int"),
])
def test_decomposed_stride_equals_undecomposed(P, Q, h, R, pad, stride, kind):
    """Stride > 1 (Sec. III-A): an input tile of Ht x Wt owns the Ht/s x Wt/s
    output block.  The decomposed passes replicate the undecomposed ones: y and
    dx bit for bit, dw within one fp32 ulp (bit for bit on integers)."""
    rng = np.random.default_rng(P * 1000 + Q * 100 + h * 10 + R + 7 * stride)
    N, C, K = 2, 3, 4
    H, W = 4 * stride * P, 3 * stride * Q
    assert orc.out_size(H, R, stride, pad) * stride == H   # output tiles align with input tiles
    x = _rand(rng, (N, C, H, W), kind)
    w = _rand(rng, (K, C, R, R), kind)
    Ho, Wo = H // stride, W // stride
    dy = _rand(rng, (N, K, Ho, Wo), kind)
    y0 = orc.round_f32(orc.conv_fwd(x, w, stride, pad))
    dx0 = orc.round_f32(orc.conv_bwd_data(dy, w, H, W, stride, pad))
    dw0 = orc.round_f32(orc.conv_bwd_filter(x, dy, R, R, stride, pad))
    y1, dx1, dw1 = (orc.round_f32(a) for a in orc.tiled_conv(x, w, dy, P, Q, h, pad, stride))
    assert np.array_equal(y0, y1)
    assert np.array_equal(dx0, dx1)
    if kind == "int":
        assert np.array_equal(dw0, dw1)
    else:
        ulp = np.abs(np.spacing(dw0))
        assert np.all(np.abs(dw0.astype(np.float64) - dw1) <= ulp)



# ------------------------------------------------- sampled-point entry points

POINT_CASES = [
    # N, C, K, H, W, R, S, stride, pad: non-square, N > 1, 1x1, 5x5, 7x7,
    # stride 2, several pads, R != S
    (3, 2, 5, 7, 9, 3, 3, 1, 1),
    (2, 3, 2, 6, 5, 1, 1, 1, 0),
    (2, 2, 3, 9, 8, 5, 5, 1, 2),
    (2, 3, 4, 11, 10, 7, 7, 2, 3),
    (1, 2, 3, 9, 7, 3, 3, 2, 1),
    (2, 2, 3, 10, 9, 3, 3, 2, 0),
    (3, 2, 2, 6, 8, 3, 5, 1, 0),
    (2, 4, 3, 8, 11, 5, 3, 1, 2),
]


def _point_indices(rng, size, n_rand=40):
    """Index 0, the last index and random indices in between."""
    return np.unique(np.concatenate([[0, size - 1], rng.integers(0, size, n_rand)])).astype(np.int64)


@pytest.mark.parametrize("case", POINT_CASES)
def test_sampled_points_equal_whole_tensor_outputs(case):
    """conv_*_points decode each flat index into (n, k|c, p|i, q|j) or
    (k, c, r, s) on their own; every sampled value must be bit-identical to
    the same element of the whole-tensor result (pinned above against a
    library convolution, finite differences and the adjoint identity) and
    agree with fp64 torch conv2d and its autograd to rounding.  A wrong decode
    order or extent (rows for columns, C for K, R for S) fails here."""
    N, C, K, H, W, R, S, st, pad = case
    rng = np.random.default_rng(abs(hash(case)) % 2**32)
    x = _rand(rng, (N, C, H, W))
    w = _rand(rng, (K, C, R, S))
    y = orc.conv_fwd(x, w, st, pad)
    dy = _rand(rng, y.shape)
    dx = orc.conv_bwd_data(dy, w, H, W, st, pad)
    dw = orc.conv_bwd_filter(x, dy, R, S, st, pad)
    xt = torch.from_numpy(x.astype(np.float64)).requires_grad_(True)
    wt = torch.from_numpy(w.astype(np.float64)).requires_grad_(True)
    yt = F.conv2d(xt, wt, stride=st, padding=pad)
    yt.backward(torch.from_numpy(dy.astype(np.float64)))
    for full, lib, pts_fn in (
            (y, yt.detach().numpy(), lambda i: orc.conv_fwd_points(x, w, st, pad, i)),
            (dx, xt.grad.numpy(), lambda i: orc.conv_bwd_data_points(dy, w, H, W, st, pad, i)),
            (dw, wt.grad.numpy(), lambda i: orc.conv_bwd_filter_points(x, dy, R, S, st, pad, i))):
        idx = _point_indices(rng, full.size)
        got = pts_fn(idx)
        assert np.array_equal(got, full.reshape(-1)[idx])
        np.testing.assert_allclose(got, lib.reshape(-1)[idx], rtol=1e-12, atol=1e-12)
        # every element once, in a shuffled order
        perm = rng.permutation(full.size).astype(np.int64)
        assert np.array_equal(pts_fn(perm), full.reshape(-1)[perm])


def test_sampled_points_of_empty_request():
    x = np.ones((1, 1, 4, 4), np.float32)
    w = np.ones((1, 1, 3, 3), np.float32)
    assert orc.conv_fwd_points(x, w, 1, 1, np.zeros(0, np.int64)).shape == (0,)
