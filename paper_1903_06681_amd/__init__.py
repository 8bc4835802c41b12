"""Python binding of libdc: one GPU's share of a spatially decomposed 2-D
convolution layer (Dryden et al., arXiv 1903.06681) on MI355X.

Argument marshalling only.  Every step of the computation runs in the HIP
kernels behind the C ABI declared in ``include/dc.h``; this module converts
torch tensors to device pointers, passes the current HIP stream and turns a
negative status into an exception.  There is no CPU fallback: importing the
package fails if ``libdc.so`` has not been built.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdc.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(
        f"{LIB_PATH} is missing: build the HIP library first "
        "(python -c 'import __graft_entry__ as g; g.build()')")

# torch brings its own HIP runtime (same soname as /opt/rocm's).  Loading it
# first makes libdc.so bind to that one copy: with the library loaded first,
# the process would hold two runtimes, and pointers and streams from torch
# would be foreign to the library's launches.
import torch  # noqa: E402,F401

_lib = ctypes.CDLL(LIB_PATH)

DC_F32, DC_BF16 = 0, 1
DC_X, DC_DY = 0, 1
DC_ALL_TILES = -1
DC_BAND_NS, DC_BAND_WE, DC_BAND_CORNERS, DC_BAND_ALL = 1, 2, 4, 7
DC_REGION_ALL, DC_REGION_INTERIOR, DC_REGION_BOUNDARY = 0, 1, 2
# capacity of the fixed workspace of dc_conv_bwd_filter_noalloc (include/dc.h)
BWD_FILTER_NOALLOC_MAX_BYTES = 64 << 20

STATUS = {
    0: "DC_OK", -1: "DC_ERR_NULL", -2: "DC_ERR_SHAPE", -3: "DC_ERR_DTYPE", -4: "DC_ERR_HALO",
    -5: "DC_ERR_UNSUPPORTED", -6: "DC_ERR_WORKSPACE", -7: "DC_ERR_ALIGN", -8: "DC_ERR_HIP",
    -9: "DC_ERR_TILE", -10: "DC_ERR_ARG", -11: "DC_ERR_TOO_LARGE",
}

EXPORTS = (
    "dc_conv_fwd", "dc_conv_bwd_data", "dc_conv_bwd_filter", "dc_halo_pack", "dc_halo_unpack",
    "dc_conv_bwd_filter_noalloc", "dc_halo_pack_bands", "dc_halo_unpack_bands",
    "dc_conv_fwd_region", "dc_conv_bwd_data_region", "dc_validate",
    "dc_tile_pitch", "dc_tile_elems", "dc_halo_elems", "dc_bwd_filter_workspace_bytes",
    "dc_required_halo", "dc_halo_bands", "dc_tile_dims", "dc_status_string",
)


class Problem(ctypes.Structure):
    """``dc_problem``: the layer (Sec. II-A) and its P x Q blocked grid (Sec. III-A)."""
    _fields_ = [(n, ctypes.c_int32) for n in
                ("N", "C", "K", "H", "W", "R", "S", "stride", "pad", "P", "Q", "halo", "dtype")]

    @classmethod
    def of(cls, layer) -> "Problem":
        """From any object with the same field names (dtype 'f32'/'bf16' or int)."""
        dt = layer.dtype
        if isinstance(dt, str):
            dt = {"f32": DC_F32, "bf16": DC_BF16}[dt]
        return cls(layer.N, layer.C, layer.K, layer.H, layer.W, layer.R, layer.S,
                   layer.stride, layer.pad, layer.P, layer.Q, layer.halo, dt)


class DcError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {STATUS.get(status, status)} "
                         f"({_lib.dc_status_string(status).decode()})")


_P = ctypes.POINTER(Problem)
_V = ctypes.c_void_p
_I = ctypes.c_int32
_lib.dc_conv_fwd.argtypes = [_P, _I, _V, _V, _V, _V]
_lib.dc_conv_bwd_data.argtypes = [_P, _I, _V, _V, _V, _V]
_lib.dc_conv_bwd_filter.argtypes = [_P, _I, _V, _V, _V, _I, _V, ctypes.c_size_t, _V]
_lib.dc_conv_bwd_filter_noalloc.argtypes = [_P, _I, _V, _V, _V, _I, _V]
_lib.dc_halo_pack.argtypes = [_P, _I, _I, _V, _V, _V]
_lib.dc_halo_unpack.argtypes = [_P, _I, _I, _V, _V, _V]
_lib.dc_conv_fwd_region.argtypes = [_P, _I, _I, _V, _V, _V, _V]
_lib.dc_conv_bwd_data_region.argtypes = [_P, _I, _I, _V, _V, _V, _V]
_lib.dc_halo_pack_bands.argtypes = [_P, _I, _I, _I, _V, _V, _V]
_lib.dc_halo_unpack_bands.argtypes = [_P, _I, _I, _I, _V, _V, _V]
_lib.dc_halo_bands.argtypes = [_P, _I, ctypes.POINTER(_I)]
_lib.dc_validate.argtypes = [_P, _I]
_lib.dc_tile_pitch.argtypes = [_P, _I]
_lib.dc_tile_pitch.restype = ctypes.c_int64
_lib.dc_tile_elems.argtypes = [_P, _I]
_lib.dc_tile_elems.restype = ctypes.c_int64
_lib.dc_halo_elems.argtypes = [_P, _I]
_lib.dc_halo_elems.restype = ctypes.c_int64
_lib.dc_bwd_filter_workspace_bytes.argtypes = [_P, _I]
_lib.dc_bwd_filter_workspace_bytes.restype = ctypes.c_size_t
_lib.dc_required_halo.argtypes = [_P, _I, ctypes.POINTER(_I)]
_lib.dc_tile_dims.argtypes = [_P, ctypes.POINTER(_I)]
_lib.dc_status_string.argtypes = [_I]
_lib.dc_status_string.restype = ctypes.c_char_p
for _n in ("dc_conv_fwd", "dc_conv_bwd_data", "dc_conv_bwd_filter", "dc_conv_bwd_filter_noalloc",
           "dc_halo_pack", "dc_halo_unpack", "dc_halo_pack_bands", "dc_halo_unpack_bands",
           "dc_conv_fwd_region", "dc_conv_bwd_data_region",
           "dc_validate", "dc_required_halo", "dc_halo_bands", "dc_tile_dims"):
    getattr(_lib, _n).restype = ctypes.c_int32


def lib():
    return _lib


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(st, where):
    if st != 0:
        raise DcError(st, where)


# ---------------------------------------------------------------- host helpers

def validate(prob: Problem, tile: int = DC_ALL_TILES) -> int:
    return _lib.dc_validate(ctypes.byref(prob), tile)


def tile_pitch(prob, which):
    return _lib.dc_tile_pitch(ctypes.byref(prob), which)


def tile_elems(prob, which):
    return _lib.dc_tile_elems(ctypes.byref(prob), which)


def halo_elems(prob, which):
    return _lib.dc_halo_elems(ctypes.byref(prob), which)


def bwd_filter_workspace_bytes(prob, tile):
    return _lib.dc_bwd_filter_workspace_bytes(ctypes.byref(prob), tile)


def required_halo(prob, which):
    out = (_I * 2)()
    _check(_lib.dc_required_halo(ctypes.byref(prob), which, out), "dc_required_halo")
    return out[0], out[1]


def halo_bands(prob, which):
    """Band widths (above, below, left, right) the halo calls move for x or dy."""
    out = (_I * 4)()
    _check(_lib.dc_halo_bands(ctypes.byref(prob), which, out), "dc_halo_bands")
    return tuple(out)


def tile_dims(prob):
    out = (_I * 4)()
    _check(_lib.dc_tile_dims(ctypes.byref(prob), out), "dc_tile_dims")
    return tuple(out)


def tile_shape(prob, which):
    """Shape [N, channels, rows + 2h, pitch] of one padded tile."""
    Ht, Wt, Hot, Wot = tile_dims(prob)
    ch = prob.C if which == DC_X else prob.K
    rows = (Ht if which == DC_X else Hot) + 2 * prob.halo
    return (prob.N, ch, rows, tile_pitch(prob, which))


# ---------------------------------------------------------------- the five calls

def conv_fwd(prob, tile, x_pad, w, y, stream=None):
    """Eq. (1) on a tile: y <- conv(x_pad, w)."""
    _check(_lib.dc_conv_fwd(ctypes.byref(prob), tile, _ptr(x_pad), _ptr(w), _ptr(y),
                            _stream(stream)), "dc_conv_fwd")


def conv_bwd_data(prob, tile, dy_pad, w, dx, stream=None):
    """Eq. (3) on a tile: dx <- input gradient from dy_pad and w."""
    _check(_lib.dc_conv_bwd_data(ctypes.byref(prob), tile, _ptr(dy_pad), _ptr(w), _ptr(dx),
                                 _stream(stream)), "dc_conv_bwd_data")


def conv_bwd_filter(prob, tile, x_pad, dy_pad, dw, accumulate, workspace, stream=None):
    """Eq. (2) on a tile: dw (=|+=) local weight gradient."""
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(_lib.dc_conv_bwd_filter(ctypes.byref(prob), tile, _ptr(x_pad), _ptr(dy_pad),
                                   _ptr(dw), accumulate, _ptr(workspace), ws_bytes,
                                   _stream(stream)), "dc_conv_bwd_filter")


def conv_bwd_filter_noalloc(prob, tile, x_pad, dy_pad, dw, accumulate, stream=None):
    """Eq. (2) on a tile with the library's fixed device workspace (no allocation)."""
    _check(_lib.dc_conv_bwd_filter_noalloc(ctypes.byref(prob), tile, _ptr(x_pad), _ptr(dy_pad),
                                           _ptr(dw), accumulate, _stream(stream)),
           "dc_conv_bwd_filter_noalloc")


def halo_pack(prob, tile, which, t_pad, send, stream=None):
    """Copy the bands neighbours need into the packed send buffer."""
    _check(_lib.dc_halo_pack(ctypes.byref(prob), tile, which, _ptr(t_pad), _ptr(send),
                             _stream(stream)), "dc_halo_pack")


def halo_unpack(prob, tile, which, recv, t_pad, stream=None):
    """Fill the margins of t_pad from the receive buffer (zeros at the domain edge)."""
    _check(_lib.dc_halo_unpack(ctypes.byref(prob), tile, which, _ptr(recv), _ptr(t_pad),
                               _stream(stream)), "dc_halo_unpack")


def halo_pack_bands(prob, tile, which, bands, t_pad, send, stream=None):
    """halo_pack restricted to the DC_BAND_* classes in `bands`."""
    _check(_lib.dc_halo_pack_bands(ctypes.byref(prob), tile, which, bands, _ptr(t_pad), _ptr(send),
                                   _stream(stream)), "dc_halo_pack_bands")


def halo_unpack_bands(prob, tile, which, bands, recv, t_pad, stream=None):
    """halo_unpack restricted to the DC_BAND_* classes in `bands`."""
    _check(_lib.dc_halo_unpack_bands(ctypes.byref(prob), tile, which, bands, _ptr(recv), _ptr(t_pad),
                                     _stream(stream)), "dc_halo_unpack_bands")


def conv_fwd_region(prob, tile, region, x_pad, w, y, stream=None):
    """Eq. (1) on the interior (no halo read) or the boundary frame of a tile."""
    _check(_lib.dc_conv_fwd_region(ctypes.byref(prob), tile, region, _ptr(x_pad), _ptr(w), _ptr(y),
                                   _stream(stream)), "dc_conv_fwd_region")


def conv_bwd_data_region(prob, tile, region, dy_pad, w, dx, stream=None):
    """Eq. (3) on the interior (no halo read) or the boundary frame of a tile."""
    _check(_lib.dc_conv_bwd_data_region(ctypes.byref(prob), tile, region, _ptr(dy_pad), _ptr(w),
                                        _ptr(dx), _stream(stream)), "dc_conv_bwd_data_region")
