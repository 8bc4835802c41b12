"""Host-side checks of libdc that need no GPU: the library loads and exports
every function include/dc.h declares, problems and arguments are validated
before anything is launched, and the tile geometry agrees with the oracle's
brute-force index sets (Sec. III-A)."""
import ctypes
import os
import re

import pytest

import oracle as orc
import paper_1903_06681_amd as dc
import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# Fake device addresses for argument-checking tests.  Every call below is
# invalid in exactly one respect that the library checks before any launch.
A16, A32, A48, MIS = 0x10000, 0x20000, 0x30000, 0x10001


def prob(**kw):
    base = dict(N=2, C=8, K=8, H=32, W=32, R=3, S=3, stride=1, pad=1, P=2, Q=2, halo=1,
                dtype=dc.DC_F32)
    base.update(kw)
    return dc.Problem(*[base[f] for f, _ in dc.Problem._fields_])


def test_every_declared_function_is_exported():
    hdr = open(os.path.join(ROOT, "include", "dc.h")).read()
    names = set(re.findall(r"\b(dc_[a-z_]+)\s*\(", hdr))
    assert {"dc_conv_fwd", "dc_conv_bwd_data", "dc_conv_bwd_filter",
            "dc_halo_pack", "dc_halo_unpack"} <= names
    lib = dc.lib()
    for n in sorted(names):
        assert hasattr(lib, n), n
    assert set(dc.EXPORTS) == names


@pytest.mark.parametrize("kw,code", [
    ({}, 0),
    ({"N": 0}, -2), ({"C": -1}, -2), ({"R": 0}, -2), ({"stride": 0}, -2), ({"pad": -1}, -2),
    ({"P": 0}, -2), ({"halo": -1}, -2),
    ({"dtype": 7}, -3),
    ({"halo": 0}, -4),                       # 3x3 needs 1
    ({"R": 5, "S": 5, "pad": 2}, -4),        # needs 2, has 1
    ({"halo": 17}, -4),                      # wider than a 16-wide tile
    ({"H": 33}, -5),                         # uneven tiles
    ({"stride": 2}, 0),                      # decomposed stride 2: 16x16 output tiles of 8
    ({"stride": 2, "H": 36, "W": 36, "P": 4, "Q": 4}, -5),   # output 18 not divisible by 4
    ({"stride": 2, "pad": 0, "halo": 2}, -5),    # output 15 * 2 != 32: grids do not line up
    ({"stride": 2, "R": 7, "S": 7, "pad": 3, "halo": 2}, -4),   # x needs 3 below
    ({"stride": 2, "R": 7, "S": 7, "pad": 3, "halo": 3}, 0),
    ({"stride": 2, "H": 16, "W": 16, "P": 4, "Q": 4, "halo": 3, "R": 7, "S": 7, "pad": 3}, -4),  # dy tile 2 < h
    ({"pad": 0, "halo": 2}, -5),             # decomposed, output not "same"
    ({"H": 2, "W": 2, "P": 1, "Q": 1, "pad": 0}, -2),  # empty output
    ({"P": 1, "Q": 1, "R": 1, "S": 1, "pad": 0, "halo": 0}, 0),
    ({"P": 1, "Q": 1, "stride": 2}, 0),
])
def test_validate_status_codes(kw, code):
    assert dc.validate(prob(**kw), dc.DC_ALL_TILES) == code


def test_tile_index_range():
    p = prob()
    assert dc.validate(p, 3) == 0
    assert dc.validate(p, 4) == -9
    assert dc.validate(p, -2) == -9


def test_all_workloads_validate():
    for L in wl.LAYERS.values():
        p = dc.Problem.of(L)
        assert dc.validate(p, dc.DC_ALL_TILES) == 0, L.name
        assert dc.tile_dims(p) == (L.Ht, L.Wt, L.Hot, L.Wot)


@pytest.mark.parametrize("R,stride,pad,H,P", [
    (3, 1, 1, 32, 2), (5, 1, 2, 40, 4), (1, 1, 0, 16, 2), (7, 2, 3, 224, 1), (3, 2, 1, 16, 1),
    (3, 2, 1, 32, 2), (7, 2, 3, 64, 4), (1, 2, 0, 16, 2), (5, 2, 2, 24, 3),
    (3, 1, 0, 12, 1), (4, 1, 1, 20, 1), (1, 2, 0, 14, 1), (5, 2, 1, 21, 1), (3, 3, 2, 17, 1),
])
def test_required_halo_matches_brute_force(R, stride, pad, H, P):
    p = prob(R=R, S=R, stride=stride, pad=pad, H=H, W=H, P=P, Q=P, halo=max(R, 3))
    lohi_x = dc.required_halo(p, dc.DC_X)
    lohi_dy = dc.required_halo(p, dc.DC_DY)
    Ho = orc.out_size(H, R, stride, pad)
    Ht, Hot = H // P, Ho // P
    bx = [0, 0]
    bd = [0, 0]
    for ti in range(P):
        lo, hi = orc.needed_halo_x(H, R, stride, pad, Ho, Ht, Hot, ti * Hot, ti * Ht)
        bx = [max(bx[0], lo), max(bx[1], hi)]
        lo, hi = orc.needed_halo_dy(Ho, R, stride, pad, Ht, Hot, ti * Ht, ti * Hot)
        bd = [max(bd[0], lo), max(bd[1], hi)]
    assert list(lohi_x) == bx
    assert list(lohi_dy) == bd


def test_one_by_one_needs_no_halo_and_packs_nothing():
    p = prob(R=1, S=1, pad=0, halo=0)
    assert dc.required_halo(p, dc.DC_X) == (0, 0)
    assert dc.halo_elems(p, dc.DC_X) == 0
    # h = 0: pack/unpack are no-ops that succeed without touching memory
    dc.halo_pack(p, dc.DC_ALL_TILES, dc.DC_X, A16, A32, 0)
    dc.halo_unpack(p, dc.DC_ALL_TILES, dc.DC_X, A16, A32, 0)


def test_empty_bands_accept_a_null_packed_buffer():
    """A margin no pass reads (1x1 filter with h = 1): every band is empty, so
    the send buffer of a pack may be NULL and nothing is launched; the tile
    pointer is still required, and a non-empty halo still requires both."""
    p = prob(R=1, S=1, pad=0, halo=1)
    assert dc.halo_elems(p, dc.DC_X) == 0 and dc.halo_elems(p, dc.DC_DY) == 0
    dc.halo_pack(p, dc.DC_ALL_TILES, dc.DC_X, A16, None, 0)
    dc.halo_pack(p, 0, dc.DC_DY, A16, None, 0)
    assert _status(dc.halo_pack, p, 0, dc.DC_X, None, None, 0) == -1
    assert _status(dc.halo_unpack, p, 0, dc.DC_X, None, None, 0) == -1
    q = prob()
    assert dc.halo_elems(q, dc.DC_X) > 0
    assert _status(dc.halo_pack, q, 0, dc.DC_X, A16, None, 0) == -1


@pytest.mark.parametrize("R,S,stride,pad,H,W,P,Q", [
    (3, 3, 1, 1, 32, 32, 2, 2), (5, 5, 1, 2, 40, 40, 4, 4), (1, 1, 1, 0, 16, 16, 2, 2),
    (7, 7, 2, 3, 224, 224, 2, 2), (3, 3, 2, 1, 32, 32, 2, 2), (7, 7, 2, 3, 64, 64, 4, 4),
    (3, 5, 1, 1, 24, 40, 1, 1), (5, 3, 2, 2, 24, 36, 1, 1), (7, 7, 2, 3, 224, 224, 1, 1),
    (5, 5, 2, 2, 24, 36, 3, 3),
])
def test_halo_bands_match_brute_force(R, S, stride, pad, H, W, P, Q):
    """Bands per side (above, below, left, right) equal the oracle's brute
    force over the index sets of Eqs. (1) and (3); halo_elems is the size of
    the eight regions they span."""
    p = prob(R=R, S=S, stride=stride, pad=pad, H=H, W=W, P=P, Q=Q, halo=max(R, S, 3) if P * Q == 1 else 3)
    if dc.validate(p, 0) != 0:
        p = prob(R=R, S=S, stride=stride, pad=pad, H=H, W=W, P=P, Q=Q, halo=max(R, S))
    assert dc.validate(p, 0) == 0
    Ht, Wt, Hot, Wot = dc.tile_dims(p)
    for which, name, ch, th, tw in ((dc.DC_X, "x", p.C, Ht, Wt), (dc.DC_DY, "dy", p.K, Hot, Wot)):
        bw = orc.halo_bands(name, H, W, R, S, stride, pad, P, Q)
        assert dc.halo_bands(p, which) == bw, name
        _, total = orc.region_offsets(p.N, ch, th, tw, p.halo, bw)
        assert dc.halo_elems(p, which) == -(-total // 4) * 4   # fp32: 16-byte multiple


def test_halo_elems_and_pitch_match_oracle_layout():
    for L in wl.LAYERS.values():
        p = dc.Problem.of(L)
        for which, name, ch, th, tw in ((dc.DC_X, "x", L.C, L.Ht, L.Wt), (dc.DC_DY, "dy", L.K, L.Hot, L.Wot)):
            bw = orc.halo_bands(name, L.H, L.W, L.R, L.S, L.stride, L.pad, L.P, L.Q)
            _, total = orc.region_offsets(L.N, ch, th, tw, L.halo, bw)
            al = 8 if L.dtype == "bf16" else 4
            assert dc.halo_elems(p, which) == -(-total // al) * al
            pitch = dc.tile_pitch(p, which)
            esize = 2 if L.dtype == "bf16" else 4
            assert pitch >= tw + 2 * L.halo and (pitch * esize) % 16 == 0
            assert dc.tile_elems(p, which) == L.N * ch * (th + 2 * L.halo) * pitch


def _status(fn, *args):
    with pytest.raises(dc.DcError) as e:
        fn(*args)
    return e.value.status


def test_calls_reject_bad_arguments_before_launch():
    p = prob()
    bad = prob(H=33)
    assert _status(dc.conv_fwd, bad, 0, A16, A32, A48, 0) == -5
    assert _status(dc.conv_fwd, p, 4, A16, A32, A48, 0) == -9
    assert _status(dc.conv_fwd, p, 0, None, A32, A48, 0) == -1
    assert _status(dc.conv_fwd, p, 0, MIS, A32, A48, 0) == -7
    assert _status(dc.conv_bwd_data, p, 0, A16, None, A48, 0) == -1
    assert _status(dc.conv_bwd_data, p, 0, A16, A32, MIS, 0) == -7
    assert _status(dc.halo_pack, p, 0, 2, A16, A32, 0) == -10
    assert _status(dc.halo_unpack, p, 0, dc.DC_X, None, A32, 0) == -1
    assert _status(dc.halo_unpack, p, 0, dc.DC_DY, A16, MIS, 0) == -7
    assert _status(dc.halo_pack_bands, p, 0, dc.DC_X, 0, A16, A32, 0) == -10
    assert _status(dc.halo_unpack_bands, p, 0, dc.DC_X, 8, A16, A32, 0) == -10


class _FakeWs:
    def __init__(self, ptr, nbytes):
        self.ptr, self.nbytes = ptr, nbytes

    def numel(self):
        return self.nbytes

    def element_size(self):
        return 1

    def data_ptr(self):
        return self.ptr


def test_bwd_filter_workspace_and_flags_checked():
    p = prob()
    need = dc.bwd_filter_workspace_bytes(p, 0)
    assert need > 0
    assert dc.bwd_filter_workspace_bytes(p, dc.DC_ALL_TILES) >= need
    assert _status(dc.conv_bwd_filter, p, 0, A16, A32, A48, 2, _FakeWs(A16, need), 0) == -10
    assert _status(dc.conv_bwd_filter, p, 0, A16, A32, A48, 0, None, 0) == -6
    assert _status(dc.conv_bwd_filter, p, 0, A16, A32, A48, 0, _FakeWs(A16, need - 4), 0) == -6
    assert _status(dc.conv_bwd_filter, p, 0, A16, A32, A48, 0, _FakeWs(MIS, need), 0) == -7
    assert _status(dc.conv_bwd_filter, p, 0, A16, None, A48, 0, _FakeWs(A16, need), 0) == -1


def test_status_strings():
    for code, name in dc.STATUS.items():
        s = dc.lib().dc_status_string(code)
        assert isinstance(s, bytes) and len(s) > 0
    assert dc.lib().dc_status_string(-99) == b"unknown status"


def test_bwd_filter_plans_only_instantiated_stride2_filters():
    """Stride-2 bf16 layers with at most 8 channels go to the phase-image
    tap-split kernel only when their phase filter (ceil(R/2) square) has an
    instantiation (2 to 4); a 9 x 9 stride-2 layer has none and must be
    rejected on the host with DC_ERR_UNSUPPORTED, not fail at launch."""
    ok = prob(N=1, C=3, K=8, H=32, W=32, R=7, S=7, stride=2, pad=3, P=1, Q=1, halo=3,
              dtype=dc.DC_BF16)
    assert dc.bwd_filter_workspace_bytes(ok, 0) > 0
    big = prob(N=1, C=3, K=8, H=32, W=32, R=9, S=9, stride=2, pad=4, P=1, Q=1, halo=4,
               dtype=dc.DC_BF16)
    assert dc.lib().dc_validate(ctypes.byref(big), 0) == 0
    assert dc.bwd_filter_workspace_bytes(big, 0) == 0
    assert _status(dc.conv_bwd_filter, big, 0, A16, A32, A48, 0, _FakeWs(A16, 1 << 20), 0) == -5


def test_noalloc_bwd_filter_limit_matches_header_and_rejects_larger_problems():
    hdr = open(os.path.join(ROOT, "include", "dc.h")).read()
    m = re.search(r"#define\s+DC_BWD_FILTER_NOALLOC_MAX_BYTES\s+\(\(size_t\)(\d+)\s*<<\s*(\d+)\)", hdr)
    assert m and int(m.group(1)) << int(m.group(2)) == dc.BWD_FILTER_NOALLOC_MAX_BYTES
    # 1024 samples of a 56x56 3x3 layer: the partials exceed the fixed array;
    # rejected on the host before the device is touched
    big = prob(N=1024, C=64, K=64, H=56, W=56, P=1, Q=1, dtype=dc.DC_BF16)
    assert dc.bwd_filter_workspace_bytes(big, 0) > dc.BWD_FILTER_NOALLOC_MAX_BYTES
    st = dc.lib().dc_conv_bwd_filter_noalloc(ctypes.byref(big), 0, A16, A32, A48, 0, None)
    assert st == -6
    p = prob()
    assert dc.lib().dc_conv_bwd_filter_noalloc(ctypes.byref(p), 0, A16, A32, A48, 2, None) == -10
    assert dc.lib().dc_conv_bwd_filter_noalloc(ctypes.byref(p), 0, A16, None, A48, 0, None) == -1
    assert dc.lib().dc_conv_bwd_filter_noalloc(ctypes.byref(p), 0, A16, A32, MIS, 0, None) == -7


def test_region_calls_checked_before_launch():
    p = prob()
    assert _status(dc.conv_fwd_region, p, 0, 3, A16, A32, A48, 0) == -10
    assert _status(dc.conv_bwd_data_region, p, 0, -1, A16, A32, A48, 0) == -10
    s2 = prob(stride=2)
    assert _status(dc.conv_fwd_region, s2, 0, dc.DC_REGION_BOUNDARY, A16, A32, A48, 0) == -5
    assert _status(dc.conv_bwd_data_region, s2, 0, dc.DC_REGION_INTERIOR, A16, A32, A48, 0) == -5
    assert _status(dc.conv_fwd_region, p, 0, dc.DC_REGION_INTERIOR, None, A32, A48, 0) == -1


def test_tiles_beyond_32bit_indexing_validate_single_samples_must_fit():
    big = prob(N=32, C=64, K=64, H=1024, W=1024, P=1, Q=1, dtype=dc.DC_BF16)
    assert dc.tile_elems(big, dc.DC_X) > 2**31          # run in groups of samples
    assert dc.validate(big, 0) == 0
    assert dc.bwd_filter_workspace_bytes(big, 0) > 0
    huge = prob(N=1, C=2048, K=64, H=1024, W=1024, P=1, Q=1, dtype=dc.DC_BF16)
    assert dc.validate(huge, 0) == -11                   # one sample alone is too large
