"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Small layers (the oracle finishes in seconds; several tiles, ragged edges)
are compared element by element, stitched over the whole grid, against the
UNDECOMPOSED oracle: Sec. III says the decomposed algorithm reproduces the
single-GPU convolution up to accumulation order.  Full-size layers run in
the single-tile launch configuration the benchmark times and are compared on
sampled outputs.  Halo pack/unpack must be bit-exact.

Tolerances: max|gpu - ref| / max|ref| <= 1e-5 for fp32 inputs and <= 2e-2 for
bf16 inputs (ref = oracle fp64 rounded once to fp32); integer-valued inputs
must agree bit for bit (every partial sum is an exact integer < 2^24).
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

TOL = {"f32": 1e-5, "bf16": 2e-2}
X, DY, ALL = dc.DC_X, dc.DC_DY, dc.DC_ALL_TILES


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()


def _rel_err(gpu, ref):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    assert np.all(np.isfinite(gpu)), "non-finite GPU output"
    denom = max(np.max(np.abs(ref)), 1e-30)
    return float(np.max(np.abs(gpu - ref)) / denom)


def _check(name, gpu, ref, dtype, exact=False):
    if exact:
        g32, r32 = np.asarray(gpu, np.float32), np.asarray(ref, np.float32)
        bad = np.argwhere(g32 != r32)
        assert bad.size == 0, (f"{name}: {len(bad)} of {g32.size} differ; first {bad[:3].tolist()}: "
                               f"{g32[tuple(bad[0])]} vs {r32[tuple(bad[0])]}")
        return 0.0
    e = _rel_err(gpu, ref)
    print(f"  {name}: max|err|/max|ref| = {e:.3e} (tol {TOL[dtype]:.0e})", flush=True)
    assert e <= TOL[dtype], (name, e)
    return e


# ------------------------------------------------------------------ layers

SMALL = {
    "c1": wl.LAYERS["c1"],
    "c2": wl.LAYERS["c2"],
    "c3a_s": wl.small("c3a", N=2, H=40, W=40),
    "c3b_s": wl.small("c3b", N=2),
    "c3c_s": wl.small("c3c", N=2, H=28, W=28),
    "c4_s": wl.small("c4", H=96, W=80, P=3, Q=2),
    "c5a_s": wl.small("c5a", N=2, H=96, W=96, P=3, Q=3),
    "c5b_s": wl.small("c5b", N=2, H=72, W=72, P=2, Q=2),
    "odd_f32": Layer("odd_f32", 2, 5, 7, 26, 39, 3, 3, 1, 1, 2, 3, 2, "f32", "uniform", 77),
    "odd_bf16": Layer("odd_bf16", 2, 5, 7, 26, 39, 3, 3, 1, 1, 2, 3, 2, "bf16", "uniform", 78),
    "k1_f32": Layer("k1_f32", 2, 6, 10, 20, 20, 1, 1, 1, 0, 2, 2, 0, "f32", "uniform", 79),
    "s2_f32": Layer("s2_f32", 2, 5, 6, 23, 23, 3, 3, 2, 1, 1, 1, 1, "f32", "uniform", 80),
    "s2k7_f32": Layer("s2k7_f32", 2, 3, 8, 30, 30, 7, 7, 2, 3, 1, 1, 3, "f32", "uniform", 81),
    "wide_bf16": Layer("wide_bf16", 1, 72, 80, 20, 150, 3, 3, 1, 1, 1, 2, 1, "bf16", "uniform", 82),
    # channel counts that leave a partial 64-wide output block in the
    # register-resident-weight kernels and a partial filter block in the
    # weight-gradient strip kernel
    "k80_bf16": Layer("k80_bf16", 2, 64, 80, 40, 40, 3, 3, 1, 1, 2, 2, 1, "bf16", "uniform", 83),
    "c32k48_bf16": Layer("c32k48_bf16", 2, 32, 48, 36, 36, 3, 3, 1, 1, 2, 2, 1, "bf16", "uniform", 84),
    "k1_48_bf16": Layer("k1_48_bf16", 2, 64, 48, 24, 24, 1, 1, 1, 0, 2, 2, 0, "bf16", "uniform", 85),
    "c48k64_bf16": Layer("c48k64_bf16", 2, 48, 64, 36, 36, 3, 3, 1, 1, 2, 2, 1, "bf16", "uniform", 86),
    # decomposed stride 2 (Sec. III-A): output tiles of Ht/2 x Wt/2, one-sided halos
    "s2dec_f32": Layer("s2dec_f32", 2, 5, 6, 32, 24, 3, 3, 2, 1, 2, 2, 1, "f32", "uniform", 87),
    "s2dec_bf16": Layer("s2dec_bf16", 2, 16, 32, 32, 32, 3, 3, 2, 1, 2, 2, 1, "bf16", "uniform", 88),
    "s2k7dec_f32": Layer("s2k7dec_f32", 1, 3, 8, 32, 32, 7, 7, 2, 3, 2, 2, 3, "f32", "uniform", 89),
    "s2k1dec_bf16": Layer("s2k1dec_bf16", 2, 32, 48, 32, 32, 1, 1, 2, 0, 2, 2, 0, "bf16", "uniform", 90),
    # at most 32 channels and filters: the weight gradient deals the taps of
    # one 32x32 block to the four waves (partial blocks, partial strips)
    "taps3_bf16": Layer("taps3_bf16", 2, 16, 24, 40, 40, 3, 3, 1, 1, 2, 2, 1, "bf16", "uniform", 91),
    "taps5_bf16": Layer("taps5_bf16", 2, 32, 20, 36, 52, 5, 5, 1, 2, 2, 2, 2, "bf16", "uniform", 92),
    "taps7_bf16": Layer("taps7_bf16", 1, 8, 32, 48, 48, 7, 7, 1, 3, 2, 2, 3, "bf16", "uniform", 93),
    # stride 2 with at most 8 channels: the weight gradient on the four phase
    # images (partial filter block, partial strips, decomposed)
    "s2taps_bf16": Layer("s2taps_bf16", 2, 5, 40, 36, 52, 5, 5, 2, 2, 2, 2, 2, "bf16", "uniform", 94),
    # stride 2 with at most 4 channels: the forward pass on the phase images
    "s2ph5_bf16": Layer("s2ph5_bf16", 2, 4, 48, 36, 52, 5, 5, 2, 2, 2, 2, 2, "bf16", "uniform", 95),
    "s2ph3_bf16": Layer("s2ph3_bf16", 2, 2, 24, 32, 32, 3, 3, 2, 1, 2, 2, 1, "bf16", "uniform", 96),
    # 3x3 on whole 32-blocks and 128-column tiles: the k-slice weight
    # gradient (two-row segments: only the guarded tail steps; and one row
    # per segment with 16-byte-aligned dy rows: halo 8, no padding)
    "kslice_bf16": Layer("kslice_bf16", 1, 32, 32, 256, 256, 3, 3, 1, 1, 2, 2, 1, "bf16", "uniform", 97),
    "kslice_p0_bf16": Layer("kslice_p0_bf16", 1, 32, 32, 130, 130, 3, 3, 1, 0, 1, 1, 8, "bf16", "uniform", 98),
    # stride 2 with at most 8 channels and 64 filters: the input gradient's
    # four output phases in one launch (7x7 window 4x4, 3x3 window 2x2;
    # decomposed, window origins not 16-byte aligned)
    "bp7_bf16": Layer("bp7_bf16", 2, 3, 64, 64, 64, 7, 7, 2, 3, 2, 2, 3, "bf16", "uniform", 99),
    "bp3_bf16": Layer("bp3_bf16", 2, 8, 64, 48, 48, 3, 3, 2, 1, 2, 2, 1, "bf16", "uniform", 100),
    # 64 channels and filters, 3x3, 128-column strips: the rolling-row forward
    # and input gradient (segments of 4 rows: rows mod 3 = 1; of 3 rows: = 0)
    "roll_bf16": Layer("roll_bf16", 1, 64, 64, 256, 256, 3, 3, 1, 1, 1, 2, 1, "bf16", "uniform", 101),
    "roll96_bf16": Layer("roll96_bf16", 2, 64, 64, 96, 128, 3, 3, 1, 1, 1, 1, 1, "bf16", "uniform", 102),
    # 32 channels and filters, 5x5: the rolling-row kernel with five live
    # output rows (segments of 8 rows: rows mod 5 = 3; of 5 rows: = 0)
    "roll5_bf16": Layer("roll5_bf16", 1, 32, 32, 256, 256, 5, 5, 1, 2, 1, 2, 2, "bf16", "uniform", 103),
    "roll5b_bf16": Layer("roll5b_bf16", 2, 32, 32, 80, 128, 5, 5, 1, 2, 1, 1, 2, "bf16", "uniform", 104),
    # the remaining tails: 3x3 segments of 5 rows (mod 3 = 2); 5x5 segments
    # of 6, 7 and 9 rows (mod 5 = 1, 2, 4)
    "roll50_bf16": Layer("roll50_bf16", 1, 64, 64, 50, 128, 3, 3, 1, 1, 1, 1, 1, "bf16", "uniform", 105),
    "roll5c_bf16": Layer("roll5c_bf16", 1, 32, 32, 96, 128, 5, 5, 1, 2, 1, 1, 2, "bf16", "uniform", 106),
    "roll5d_bf16": Layer("roll5d_bf16", 1, 32, 32, 112, 128, 5, 5, 1, 2, 1, 1, 2, "bf16", "uniform", 107),
    "roll5e_bf16": Layer("roll5e_bf16", 1, 32, 32, 81, 128, 5, 5, 1, 2, 1, 1, 2, "bf16", "uniform", 108),
    # fp32 register-weight kernels below their channel capacity class (4, 8,
    # .., 32 and 18): channel counts between the classes, odd ones included,
    # for the forward (C), the input gradient (K) and the weight gradient
    "f32_c3": Layer("f32_c3", 2, 3, 12, 34, 30, 3, 3, 1, 1, 2, 2, 1, "f32", "uniform", 109),
    "f32_c13": Layer("f32_c13", 2, 13, 20, 40, 36, 3, 3, 1, 1, 2, 2, 1, "f32", "uniform", 110),
    "f32_c17": Layer("f32_c17", 1, 17, 30, 48, 40, 3, 3, 1, 1, 2, 2, 1, "f32", "uniform", 111),
    "f32_c29": Layer("f32_c29", 1, 29, 7, 36, 36, 3, 3, 1, 1, 2, 2, 1, "f32", "uniform", 112),
    "k1_c22_f32": Layer("k1_c22_f32", 2, 22, 11, 24, 20, 1, 1, 1, 0, 2, 2, 0, "f32", "uniform", 113),
    # the ends of the classes: one channel (class 4), and 36 / 40 channels,
    # past the largest class, on the chunked and row kernels instead
    "f32_c1": Layer("f32_c1", 2, 1, 3, 20, 24, 3, 3, 1, 1, 2, 2, 1, "f32", "uniform", 114),
    "f32_c36": Layer("f32_c36", 1, 36, 40, 24, 24, 3, 3, 1, 1, 2, 2, 1, "f32", "uniform", 115),
    # a single filter (K = 1): one-channel input-gradient reduction, one-row weight gradient
    "k_one": Layer("k_one", 2, 16, 1, 24, 40, 3, 3, 1, 1, 2, 2, 1, "bf16", "uniform", 116),
    "k_one_f32": Layer("k_one_f32", 2, 5, 1, 20, 28, 3, 3, 1, 1, 2, 2, 1, "f32", "uniform", 117),
}


def _gpu_all_tiles(L, x, w, dy):
    """Whole grid in all-tiles launches: halos, fwd, bwd-data, bwd-filter."""
    p = dc.Problem.of(L)
    nt = L.P * L.Q
    xt = H.alloc_tiles(p, X, nt, L.dtype)
    dyt = H.alloc_tiles(p, DY, nt, L.dtype)
    H.scatter_interiors(xt, H.to_device(x, L.dtype), p, X)
    H.scatter_interiors(dyt, H.to_device(dy, L.dtype), p, DY)
    H.fill_halos_all_tiles(p, X, xt, L.dtype)
    H.fill_halos_all_tiles(p, DY, dyt, L.dtype)
    wd = H.to_device(w, L.dtype)
    y = torch.full((nt, L.N, L.K, L.Hot, L.Wot), float("nan"), device="cuda")
    dx = torch.full((nt, L.N, L.C, L.Ht, L.Wt), float("nan"), device="cuda")
    dw = torch.full((L.K, L.C, L.R, L.S), float("nan"), device="cuda")
    ws = torch.empty(max(dc.bwd_filter_workspace_bytes(p, ALL), 16), dtype=torch.uint8, device="cuda")
    dc.conv_fwd(p, ALL, xt, wd, y)
    dc.conv_bwd_data(p, ALL, dyt, wd, dx)
    dc.conv_bwd_filter(p, ALL, xt, dyt, dw, 0, ws)
    torch.cuda.synchronize()
    yg = H.gather_outputs(y, p, "y").cpu().numpy()
    dxg = H.gather_outputs(dx, p, "dx").cpu().numpy()
    return yg, dxg, dw.cpu().numpy(), (xt, dyt, wd, ws)


def _oracle_full(L, x, w, dy):
    y = orc.round_f32(orc.conv_fwd(x, w, L.stride, L.pad))
    dx = orc.round_f32(orc.conv_bwd_data(dy, w, L.H, L.W, L.stride, L.pad))
    dw = orc.round_f32(orc.conv_bwd_filter(x, dy, L.R, L.S, L.stride, L.pad))
    return y, dx, dw


@pytest.mark.parametrize("name", list(SMALL))
def test_small_layer_all_tiles_matches_undecomposed_oracle(name):
    L = SMALL[name]
    print(f"[parity] {name}: {L}", flush=True)
    x, w, dy = wl.draw(L, "x"), wl.draw(L, "w"), wl.draw(L, "dy")
    yg, dxg, dwg, _ = _gpu_all_tiles(L, x, w, dy)
    yr, dxr, dwr = _oracle_full(L, x, w, dy)
    assert yg.shape == yr.shape and dxg.shape == dxr.shape
    _check("y", yg, yr, L.dtype)
    _check("dx", dxg, dxr, L.dtype)
    _check("dw", dwg, dwr, L.dtype)


@pytest.mark.parametrize("name", ["c2", "odd_f32", "odd_bf16", "c5a_s", "c5b_s", "s2k7_f32", "c3a_s",
                                  "k80_bf16", "c48k64_bf16", "s2dec_bf16", "s2k7dec_f32", "taps5_bf16", "s2taps_bf16",
                                  "s2ph5_bf16", "kslice_bf16", "kslice_p0_bf16", "bp7_bf16", "bp3_bf16",
                                  "roll_bf16", "roll96_bf16", "roll5_bf16", "roll5b_bf16",
                                  "roll50_bf16", "roll5c_bf16", "roll5d_bf16", "roll5e_bf16",
                                  "f32_c3", "f32_c17", "k1_c22_f32", "f32_c1", "f32_c36", "k_one",
                                  "k_one_f32"])
def test_integer_inputs_are_bit_exact(name):
    """Integer data in {-2..2}: all sums are exact integers, whatever the order."""
    L = SMALL[name]
    print(f"[exact] {name}", flush=True)
    x, w, dy = (wl.draw(L, t, dist="int") for t in ("x", "w", "dy"))
    yg, dxg, dwg, _ = _gpu_all_tiles(L, x, w, dy)
    yr, dxr, dwr = _oracle_full(L, x, w, dy)
    _check("y", yg, yr, L.dtype, exact=True)
    _check("dx", dxg, dxr, L.dtype, exact=True)
    _check("dw", dwg, dwr, L.dtype, exact=True)


@pytest.mark.parametrize("name", ["c2", "odd_bf16", "c5b_s", "s2k7dec_f32", "taps7_bf16"])
def test_single_tile_calls_match_all_tiles(name):
    """Per-tile pack -> emulated exchange (region copies) -> unpack -> passes
    equals the all-tiles launch bit for bit, and accumulate=1 sums the tiles."""
    L = SMALL[name]
    p = dc.Problem.of(L)
    nt = L.P * L.Q
    x, w, dy = wl.draw(L, "x"), wl.draw(L, "w"), wl.draw(L, "dy")
    yg, dxg, dwg, (xt_all, dyt_all, wd, _) = _gpu_all_tiles(L, x, w, dy)
    xg, dyg = H.to_device(x, L.dtype), H.to_device(dy, L.dtype)
    # interiors only; sends of every tile packed one call at a time
    xt = H.alloc_tiles(p, X, nt, L.dtype)
    dyt = H.alloc_tiles(p, DY, nt, L.dtype)
    H.scatter_interiors(xt, xg, p, X)
    H.scatter_interiors(dyt, dyg, p, DY)
    tdt = H.TORCH_DT[L.dtype]
    sx = torch.zeros((nt, dc.halo_elems(p, X)), dtype=tdt, device="cuda")
    sy = torch.zeros((nt, dc.halo_elems(p, DY)), dtype=tdt, device="cuda")
    for t in range(nt):
        dc.halo_pack(p, t, X, xt[t], sx[t])
        dc.halo_pack(p, t, DY, dyt[t], sy[t])
    dw = torch.zeros((L.K, L.C, L.R, L.S), device="cuda")
    ws = torch.empty(dc.bwd_filter_workspace_bytes(p, 0), dtype=torch.uint8, device="cuda")
    for t in range(nt):
        rx = torch.zeros_like(sx[t])
        ry = torch.zeros_like(sy[t])
        H.exchange_into(rx, sx, p, X, t)
        H.exchange_into(ry, sy, p, DY, t)
        dc.halo_unpack(p, t, X, rx, xt[t])
        dc.halo_unpack(p, t, DY, ry, dyt[t])
        assert torch.equal(xt[t].view(torch.int16 if L.dtype == "bf16" else torch.int32),
                           xt_all[t].view(torch.int16 if L.dtype == "bf16" else torch.int32))
        y = torch.empty((L.N, L.K, L.Hot, L.Wot), device="cuda")
        dx = torch.empty((L.N, L.C, L.Ht, L.Wt), device="cuda")
        dc.conv_fwd(p, t, xt[t], wd, y)
        dc.conv_bwd_data(p, t, dyt[t], wd, dx)
        dc.conv_bwd_filter(p, t, xt[t], dyt[t], dw, 1 if t > 0 else 0, ws)
        ti, tj = divmod(t, L.Q)
        assert np.array_equal(y.cpu().numpy(),
                              yg[:, :, ti * L.Hot:(ti + 1) * L.Hot, tj * L.Wot:(tj + 1) * L.Wot])
        assert np.array_equal(dx.cpu().numpy(),
                              dxg[:, :, ti * L.Ht:(ti + 1) * L.Ht, tj * L.Wt:(tj + 1) * L.Wt])
    torch.cuda.synchronize()
    yr, dxr, dwr = _oracle_full(L, x, w, dy)
    _check("dw (sum of per-tile partials)", dw.cpu().numpy(), dwr, L.dtype)


# ------------------------------------------------------------------ halos

def _bits(t):
    return t.view(torch.int16 if t.dtype == torch.bfloat16 else torch.int32).cpu().numpy()


def _oracle_bands(L, which):
    return orc.halo_bands("x" if which == X else "dy", L.H, L.W, L.R, L.S, L.stride, L.pad, L.P, L.Q)


@pytest.mark.parametrize("name", ["c2", "odd_f32", "odd_bf16", "c5b_s", "c4_s", "s2dec_bf16",
                                  "s2k7dec_f32", "bp7_bf16", "s2taps_bf16", "wide_bf16"])
@pytest.mark.parametrize("which", [X, DY])
def test_halo_pack_unpack_bit_exact(name, which):
    """Bands per side (one-sided at stride 2, narrower than the margin for
    odd_*), margins beyond the bands zeroed, pitch columns never written."""
    L = SMALL[name]
    p = dc.Problem.of(L)
    nt = L.P * L.Q
    g = wl.draw(L, "x" if which == X else "dy")
    ch = L.C if which == X else L.K
    th, tw = (L.Ht, L.Wt) if which == X else (L.Hot, L.Wot)
    gh, gw = g.shape[2], g.shape[3]
    tiles = H.alloc_tiles(p, which, nt, L.dtype)
    H.scatter_interiors(tiles, H.to_device(g, L.dtype), p, which)
    hel = dc.halo_elems(p, which)
    sentinel = -3.0   # exact in bf16 and fp32; regions without a neighbour keep it
    send = torch.full((nt, hel), sentinel, dtype=H.TORCH_DT[L.dtype], device="cuda")
    dc.halo_pack(p, ALL, which, tiles, send)
    dc.halo_unpack(p, ALL, which, send, tiles)
    torch.cuda.synchronize()
    sb, tb = _bits(send), _bits(tiles)
    h = L.halo
    bw = _oracle_bands(L, which)
    gq = g if L.dtype == "f32" else g  # values already bf16-representable
    for t in range(nt):
        ti, tj = divmod(t, L.Q)
        # pack: regions with a neighbour equal the oracle's; the rest untouched (NaN)
        ref = np.full(hel, sentinel, np.float32)
        ntot = orc.region_offsets(L.N, L.C if which == X else L.K, *((L.Ht, L.Wt) if which == X else (L.Hot, L.Wot)), h, bw)[1]
        orc.halo_pack(gq, L.P, L.Q, ti, tj, h, ref[:ntot], bw)   # padding to 16 bytes stays untouched
        rb = _bits(H.to_device(ref, L.dtype))
        bad = np.nonzero(sb[t] != rb)[0]
        assert bad.size == 0, f"pack tile {t}: {bad.size} mismatches, first at {bad[:5]}: {sb[t][bad[:5]]} vs {rb[bad[:5]]}"
        # unpack: the window equals the zero-padded global slice; pitch columns untouched
        win = orc.tile_window(gq, L.P, L.Q, ti, tj, h, bw)
        wb = _bits(H.to_device(win, L.dtype))
        got = tb[t][:, :, :, :tw + 2 * h]
        bad = np.argwhere(got != wb)
        assert bad.size == 0, f"unpack tile {t}: {len(bad)} mismatches, first {bad[:5].tolist()}"
        pad_cols = tiles[t][:, :, :, tw + 2 * h:]
        assert bool(torch.isnan(pad_cols.float()).all()), "pitch padding written"


@pytest.mark.parametrize("name", ["c5b_s", "odd_bf16", "s2dec_bf16", "c4_s"])
@pytest.mark.parametrize("which", [X, DY])
def test_halo_band_classes_compose_to_the_full_calls(name, which):
    """Pack and unpack by band class (N/S rows, W/E columns, corners), one
    class per call, give the full calls' bits; each class writes only its
    own regions (pack) and its own margin cells (unpack)."""
    L = SMALL[name]
    p = dc.Problem.of(L)
    nt = L.P * L.Q
    g = wl.draw(L, "x" if which == X else "dy")
    tiles = H.alloc_tiles(p, which, nt, L.dtype)
    H.scatter_interiors(tiles, H.to_device(g, L.dtype), p, which)
    hel = dc.halo_elems(p, which)
    tdt = H.TORCH_DT[L.dtype]
    full = torch.full((nt, hel), -3.0, dtype=tdt, device="cuda")
    parts = torch.full((nt, hel), -3.0, dtype=tdt, device="cuda")
    dc.halo_pack(p, ALL, which, tiles, full)
    table = H.region_table(p, which, send=True)
    cls = {dc.DC_BAND_NS: ("N", "S"), dc.DC_BAND_WE: ("W", "E"),
           dc.DC_BAND_CORNERS: ("NW", "NE", "SW", "SE")}
    ch = L.C if which == X else L.K
    for band, dirs in cls.items():
        before = parts.clone()
        dc.halo_pack_bands(p, ALL, which, band, tiles, parts)
        torch.cuda.synchronize()
        changed = (_bits(parts) != _bits(before))
        for d, (off, r, c) in table.items():
            if d not in dirs:
                assert not changed[:, off:off + L.N * ch * r * c].any(), (band, d)
    assert np.array_equal(_bits(parts), _bits(full))
    # unpack: the full call vs one class at a time, both into NaN margins
    t_full = tiles.clone()
    t_parts = tiles.clone()
    dc.halo_unpack(p, ALL, which, full, t_full)
    h = L.halo
    th, tw = (L.Ht, L.Wt) if which == X else (L.Hot, L.Wot)
    rows = np.arange(th + 2 * h)[:, None]
    cols = np.arange(tw + 2 * h)[None, :]
    rin, cin = (rows >= h) & (rows < h + th), (cols >= h) & (cols < h + tw)
    cells = {dc.DC_BAND_NS: ~rin & cin, dc.DC_BAND_WE: rin & ~cin, dc.DC_BAND_CORNERS: ~rin & ~cin}
    for band, mask in cells.items():
        before = _bits(t_parts).copy()
        dc.halo_unpack_bands(p, ALL, which, band, full, t_parts)
        torch.cuda.synchronize()
        after = _bits(t_parts)
        diff = (after != before)[..., :tw + 2 * h].any(axis=(0, 1, 2))
        assert not (diff & ~mask).any(), band
    assert np.array_equal(_bits(t_parts), _bits(t_full))


def test_unpack_writes_only_margins():
    L = SMALL["c2"]
    p = dc.Problem.of(L)
    nt = L.P * L.Q
    tiles = torch.full((nt,) + dc.tile_shape(p, X), 7.0, device="cuda")
    send = torch.full((nt, dc.halo_elems(p, X)), -3.0, device="cuda")
    dc.halo_unpack(p, ALL, X, send, tiles)
    torch.cuda.synchronize()
    h, Ht, Wt = L.halo, L.Ht, L.Wt
    inner = tiles[:, :, :, h:h + Ht, h:h + Wt]
    assert bool((inner == 7.0).all())
    pad = tiles[:, :, :, :, Wt + 2 * h:]
    assert bool((pad == 7.0).all())


# ------------------------------------------------------------------ properties

def test_stale_hip_error_of_the_caller_is_not_reported():
    """hipGetLastError keeps the last error of any earlier HIP call: an error
    the caller left behind must not make the next library call fail.  Each
    call below runs right after an invalid hipSetDevice has set that error."""
    import ctypes
    hip = ctypes.CDLL("libamdhip64.so")

    def stale():
        assert hip.hipSetDevice(ctypes.c_int(1 << 20)) != 0   # invalid ordinal

    L = SMALL["odd_bf16"]
    p = dc.Problem.of(L)
    nt = L.P * L.Q
    x, w, dy = (wl.draw(L, t) for t in ("x", "w", "dy"))
    xt = H.alloc_tiles(p, X, nt, L.dtype)
    dyt = H.alloc_tiles(p, DY, nt, L.dtype)
    H.scatter_interiors(xt, H.to_device(x, L.dtype), p, X)
    H.scatter_interiors(dyt, H.to_device(dy, L.dtype), p, DY)
    wd = H.to_device(w, L.dtype)
    y = torch.empty((nt, L.N, L.K, L.Hot, L.Wot), device="cuda")
    dx = torch.empty((nt, L.N, L.C, L.Ht, L.Wt), device="cuda")
    dw = torch.empty((L.K, L.C, L.R, L.S), device="cuda")
    ws = torch.empty(max(dc.bwd_filter_workspace_bytes(p, ALL), 16), dtype=torch.uint8, device="cuda")
    sx = torch.empty(nt * dc.halo_elems(p, X), dtype=H.TORCH_DT[L.dtype], device="cuda")
    sdy = torch.empty(nt * dc.halo_elems(p, DY), dtype=H.TORCH_DT[L.dtype], device="cuda")
    torch.cuda.synchronize()
    for f in (lambda: dc.halo_pack(p, ALL, X, xt, sx), lambda: dc.halo_unpack(p, ALL, X, sx, xt),
              lambda: dc.halo_pack(p, ALL, DY, dyt, sdy), lambda: dc.halo_unpack(p, ALL, DY, sdy, dyt),
              lambda: dc.conv_fwd(p, ALL, xt, wd, y), lambda: dc.conv_bwd_data(p, ALL, dyt, wd, dx),
              lambda: dc.conv_bwd_filter(p, ALL, xt, dyt, dw, 0, ws)):
        stale()
        f()
    hip.hipGetLastError()
    torch.cuda.synchronize()
    yr, dxr, dwr = _oracle_full(L, x, w, dy)
    _check("y", H.gather_outputs(y, p, "y").cpu().numpy(), yr, L.dtype)
    _check("dx", H.gather_outputs(dx, p, "dx").cpu().numpy(), dxr, L.dtype)
    _check("dw", dw.cpu().numpy(), dwr, L.dtype)


@pytest.mark.parametrize("name", ["c5a_s", "kslice_bf16", "kslice_p0_bf16", "taps5_bf16", "c4_s"])
def test_bwd_filter_ignores_dy_halo_and_is_deterministic(name):
    """dw needs no dy halo (Sec. III-A): NaN in every dy margin must not reach
    dw.  Two runs give identical bits (fixed-order reduction, no atomics).
    kslice_* run the k-slice kernel, whose 16-byte dy loads start on the
    margin column."""
    L = SMALL[name]
    p = dc.Problem.of(L)
    nt = L.P * L.Q
    x, w, dy = wl.draw(L, "x"), wl.draw(L, "w"), wl.draw(L, "dy")
    xt = H.alloc_tiles(p, X, nt, L.dtype)
    dyt = H.alloc_tiles(p, DY, nt, L.dtype)   # margins stay NaN
    H.scatter_interiors(xt, H.to_device(x, L.dtype), p, X)
    H.scatter_interiors(dyt, H.to_device(dy, L.dtype), p, DY)
    H.fill_halos_all_tiles(p, X, xt, L.dtype)
    ws = torch.empty(dc.bwd_filter_workspace_bytes(p, ALL), dtype=torch.uint8, device="cuda")
    dw1 = torch.empty((L.K, L.C, L.R, L.S), device="cuda")
    dw2 = torch.empty_like(dw1)
    dc.conv_bwd_filter(p, ALL, xt, dyt, dw1, 0, ws)
    dc.conv_bwd_filter(p, ALL, xt, dyt, dw2, 0, ws)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(dw1).all())
    assert torch.equal(dw1.view(torch.int32), dw2.view(torch.int32))
    dwr = orc.round_f32(orc.conv_bwd_filter(x, dy, L.R, L.S, L.stride, L.pad))
    _check("dw", dw1.cpu().numpy(), dwr, L.dtype)


# ------------------------------------------------------------------ full size

def _seam_lines(lo, hi, period):
    """Lines lo <= v < hi on either side of every multiple of `period` past lo."""
    out = []
    for m in range(lo + period, hi, period):
        out += [m - 1, m]
    return np.array(out, np.int64)


def _sample_idx(rng, shape, region, n_rand, edges=True, seams=True):
    """Flat indices into a tensor of `shape` = [A, B, rows, cols], restricted to
    rows/cols in region=(r0, r1, c0, c1), including the region's border lines
    and, with seams, the lines on both sides of every 8-row boundary (row
    segments of the rolling-row and k-slice kernels) and every 64-column
    boundary (64- and 128-column strips), where work passes from one
    workgroup to the next."""
    A, B, Hh, Ww = shape
    r0, r1, c0, c1 = region
    pts = []
    if seams:
        sr, sc = _seam_lines(r0, r1, 8), _seam_lines(c0, c1, 64)
        m = n_rand // 4
        if sr.size:
            pts.append(np.stack([rng.integers(0, A, m), rng.integers(0, B, m),
                                 rng.choice(sr, m), rng.integers(c0, c1, m)], 1))
        if sc.size:
            pts.append(np.stack([rng.integers(0, A, m), rng.integers(0, B, m),
                                 rng.integers(r0, r1, m), rng.choice(sc, m)], 1))
        if sr.size and sc.size:
            pts.append(np.stack([rng.integers(0, A, m), rng.integers(0, B, m),
                                 rng.choice(sr, m), rng.choice(sc, m)], 1))
    a = rng.integers(0, A, n_rand)
    b = rng.integers(0, B, n_rand)
    r = rng.integers(r0, r1, n_rand)
    c = rng.integers(c0, c1, n_rand)
    pts.append(np.stack([a, b, r, c], 1))
    if edges:
        m = n_rand // 4
        for rr in (r0, r1 - 1):
            pts.append(np.stack([rng.integers(0, A, m), rng.integers(0, B, m),
                                 np.full(m, rr), rng.integers(c0, c1, m)], 1))
        for cc in (c0, c1 - 1):
            pts.append(np.stack([rng.integers(0, A, m), rng.integers(0, B, m),
                                 rng.integers(r0, r1, m), np.full(m, cc)], 1))
        for rr in (r0, r1 - 1):
            for cc in (c0, c1 - 1):
                pts.append(np.stack([rng.integers(0, A, 8), rng.integers(0, B, 8),
                                     np.full(8, rr), np.full(8, cc)], 1))
    P = np.concatenate(pts, 0)
    flat = ((P[:, 0] * B + P[:, 1]) * Hh + P[:, 2]) * Ww + P[:, 3]
    return flat.astype(np.int64), P


FULL = [("c5a", 5), ("c5a", 0), ("c5b", 5), ("c5b", 0), ("c4", 5), ("c4", 0),
        ("c3a", 0), ("c3b", 0), ("c3c", 0), ("c3a_2x2", 3), ("c3a_2x2", 0), ("c4s2", 5), ("c4s2", 0)]


@pytest.mark.parametrize("name,tile", FULL)
def test_full_size_single_tile_sampled(name, tile):
    """Full-size layer, one tile, single-tile launches (the benchmark's
    configuration), sampled against the undecomposed oracle (y, dx) and the
    oracle's per-tile weight-gradient sum (dw)."""
    L = wl.LAYERS[name]
    p = dc.Problem.of(L)
    print(f"[full] {name} tile {tile}: {L.desc}", flush=True)
    rng = np.random.default_rng(1234 + tile)
    x, w, dy = wl.draw(L, "x"), wl.draw(L, "w"), wl.draw(L, "dy")
    nt = L.P * L.Q
    ti, tj = divmod(tile, L.Q)
    tdt = H.TORCH_DT[L.dtype]
    # neighbours' sends: pack every tile (all-tiles launch), then the exchange
    # copies this tile's receive buffer from them
    xt = H.alloc_tiles(p, X, nt, L.dtype)
    dyt = H.alloc_tiles(p, DY, nt, L.dtype)
    H.scatter_interiors(xt, H.to_device(x, L.dtype), p, X)
    H.scatter_interiors(dyt, H.to_device(dy, L.dtype), p, DY)
    sx = torch.empty((nt, max(dc.halo_elems(p, X), 1)), dtype=tdt, device="cuda")
    sy = torch.empty((nt, max(dc.halo_elems(p, DY), 1)), dtype=tdt, device="cuda")
    dc.halo_pack(p, ALL, X, xt, sx)
    dc.halo_pack(p, ALL, DY, dyt, sy)
    rx, ry = torch.zeros_like(sx[0]), torch.zeros_like(sy[0])
    H.exchange_into(rx, sx, p, X, tile)
    H.exchange_into(ry, sy, p, DY, tile)
    xme, dyme = xt[tile].clone(), dyt[tile].clone()
    del xt, dyt
    dc.halo_unpack(p, tile, X, rx, xme)
    dc.halo_unpack(p, tile, DY, ry, dyme)
    wd = H.to_device(w, L.dtype)
    y = torch.empty((L.N, L.K, L.Hot, L.Wot), device="cuda")
    dx = torch.empty((L.N, L.C, L.Ht, L.Wt), device="cuda")
    dw = torch.empty((L.K, L.C, L.R, L.S), device="cuda")
    ws = torch.empty(dc.bwd_filter_workspace_bytes(p, tile), dtype=torch.uint8, device="cuda")
    dc.conv_fwd(p, tile, xme, wd, y)
    dc.conv_bwd_data(p, tile, dyme, wd, dx)
    dc.conv_bwd_filter(p, tile, xme, dyme, dw, 0, ws)
    torch.cuda.synchronize()
    y, dx, dw = y.cpu().numpy(), dx.cpu().numpy(), dw.cpu().numpy()
    assert np.all(np.isfinite(y)) and np.all(np.isfinite(dx)) and np.all(np.isfinite(dw))

    # y at sampled global outputs of this tile (undecomposed Eq. (1))
    region = (ti * L.Hot, (ti + 1) * L.Hot, tj * L.Wot, (tj + 1) * L.Wot)
    flat, P = _sample_idx(rng, (L.N, L.K, L.Ho, L.Wo), region, 1024)
    ref = orc.round_f32(orc.conv_fwd_points(x, w, L.stride, L.pad, flat))
    got = y[P[:, 0], P[:, 1], P[:, 2] - region[0], P[:, 3] - region[2]]
    _check("y (sampled)", got, ref, L.dtype)
    # dx at sampled global inputs of this tile (undecomposed Eq. (3))
    region = (ti * L.Ht, (ti + 1) * L.Ht, tj * L.Wt, (tj + 1) * L.Wt)
    flat, P = _sample_idx(rng, (L.N, L.C, L.H, L.W), region, 1024)
    ref = orc.round_f32(orc.conv_bwd_data_points(dy, w, L.H, L.W, L.stride, L.pad, flat))
    got = dx[P[:, 0], P[:, 1], P[:, 2] - region[0], P[:, 3] - region[2]]
    _check("dx (sampled)", got, ref, L.dtype)
    # local dw: Eq. (2) over this tile's samples and output pixels only
    if L.P * L.Q == 1:
        xs, dys, pad = x, dy, L.pad
    else:
        # the x rows/cols the tile's outputs reach: from -pad, (Hot-1)*stride + R of them
        nr, ns = (L.Hot - 1) * L.stride + L.R, (L.Wot - 1) * L.stride + L.S
        win = orc.tile_window(x, L.P, L.Q, ti, tj, L.halo)
        h = L.halo
        xs = np.ascontiguousarray(win[:, :, h - L.pad:h - L.pad + nr, h - L.pad:h - L.pad + ns])
        dys = np.ascontiguousarray(dy[:, :, ti * L.Hot:(ti + 1) * L.Hot, tj * L.Wot:(tj + 1) * L.Wot])
        pad = 0
    n_dw = min(256, dw.size)
    flat = rng.choice(dw.size, n_dw, replace=False).astype(np.int64)
    ref = orc.round_f32(orc.conv_bwd_filter_points(xs, dys, L.R, L.S, L.stride, pad, flat))
    _check("dw local (sampled)", dw.reshape(-1)[flat], ref, L.dtype)
