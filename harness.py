"""GPU-side plumbing shared by the tests, the benchmark and the smoke check.

Allocates padded tiles in the library's layout, scatters a global tensor's
owned blocks into tile interiors, gathers tile outputs back into a global
tensor, and emulates the halo transport for single-tile calls by copying the
neighbours' packed regions (torch device copies).  It holds no convolution
arithmetic and never imports the oracle.
"""
from __future__ import annotations

import numpy as np
import torch

import paper_1903_06681_amd as dc

TORCH_DT = {"f32": torch.float32, "bf16": torch.bfloat16}
DIRS = ("N", "S", "W", "E", "NW", "NE", "SW", "SE")
STEP = {"N": (-1, 0), "S": (1, 0), "W": (0, -1), "E": (0, 1),
        "NW": (-1, -1), "NE": (-1, 1), "SW": (1, -1), "SE": (1, 1)}
OPP = {"N": "S", "S": "N", "W": "E", "E": "W", "NW": "SE", "NE": "SW", "SW": "NE", "SE": "NW"}


def to_device(a: np.ndarray, dtype: str, device="cuda") -> torch.Tensor:
    """fp32 numpy values (bf16-representable for bf16) -> device tensor of the layer dtype."""
    t = torch.from_numpy(np.ascontiguousarray(a))
    return t.to(device=device, dtype=TORCH_DT[dtype])


def alloc_tiles(prob, which, ntiles, dtype, device="cuda", fill=float("nan")):
    shape = (ntiles,) + dc.tile_shape(prob, which)
    return torch.full(shape, fill, dtype=TORCH_DT[dtype], device=device)


def scatter_interiors(tiles: torch.Tensor, g: torch.Tensor, prob, which, tile_ids=None):
    """tiles[t, :, :, h:h+Ht, h:h+Wt] = owned block of tile t in the global g [N, ch, H, W]."""
    Ht, Wt, Hot, Wot = dc.tile_dims(prob)
    th, tw = (Ht, Wt) if which == dc.DC_X else (Hot, Wot)
    h = prob.halo
    ids = range(prob.P * prob.Q) if tile_ids is None else tile_ids
    for k, t in enumerate(ids):
        ti, tj = divmod(t, prob.Q)
        dst = tiles[k] if tile_ids is not None else tiles[t]
        dst[:, :, h:h + th, h:h + tw] = g[:, :, ti * th:(ti + 1) * th, tj * tw:(tj + 1) * tw]


def gather_outputs(out_tiles: torch.Tensor, prob, which_out: str) -> torch.Tensor:
    """Stitch per-tile outputs [ntiles, N, ch, th, tw] into [N, ch, P*th, Q*tw]."""
    nt, N, ch, th, tw = out_tiles.shape
    g = out_tiles.new_empty((N, ch, prob.P * th, prob.Q * tw))
    for t in range(nt):
        ti, tj = divmod(t, prob.Q)
        g[:, :, ti * th:(ti + 1) * th, tj * tw:(tj + 1) * tw] = out_tiles[t]
    return g


def region_table(prob, which, send=False):
    """(offset, rows, cols) of each packed region, in the interface's fixed
    order: receive regions have the shape of the tile's margin bands, send
    regions that of the neighbour's opposite margin band."""
    Ht, Wt, Hot, Wot = dc.tile_dims(prob)
    th, tw = (Ht, Wt) if which == dc.DC_X else (Hot, Wot)
    ch = prob.C if which == dc.DC_X else prob.K
    bn, bs, bw, be = dc.halo_bands(prob, which)
    rows = {-1: bn, 0: th, 1: bs}
    cols = {-1: bw, 0: tw, 1: be}
    table, off = {}, 0
    for d in DIRS:
        di, dj = STEP[OPP[d]] if send else STEP[d]
        r, c = rows[di], cols[dj]
        table[d] = (off, r, c)
        off += prob.N * ch * r * c
    return table


def neighbour(prob, t, d):
    ti, tj = divmod(t, prob.Q)
    ni, nj = ti + STEP[d][0], tj + STEP[d][1]
    if 0 <= ni < prob.P and 0 <= nj < prob.Q:
        return ni * prob.Q + nj
    return None


def exchange_into(recv: torch.Tensor, sends: torch.Tensor, prob, which, t):
    """Emulated transport for tile t: recv region d <- neighbour d's region opposite(d).
    sends: [ntiles, halo_elems] packed buffers of all tiles; recv: [halo_elems]."""
    table = region_table(prob, which)
    stable = region_table(prob, which, send=True)
    for d in DIRS:
        nb = neighbour(prob, t, d)
        if nb is None:
            continue
        off, r, c = table[d]
        ooff = stable[OPP[d]][0]
        ch = prob.C if which == dc.DC_X else prob.K
        n = prob.N * ch * r * c
        recv[off:off + n].copy_(sends[nb, ooff:ooff + n])


def fill_halos_all_tiles(prob, which, tiles, dtype):
    """pack (all tiles) + unpack (all tiles, reading neighbours' sends directly)."""
    hel = dc.halo_elems(prob, which)
    send = torch.empty((prob.P * prob.Q, max(hel, 1)), dtype=TORCH_DT[dtype], device=tiles.device)
    dc.halo_pack(prob, dc.DC_ALL_TILES, which, tiles, send)
    dc.halo_unpack(prob, dc.DC_ALL_TILES, which, send, tiles)
    return send
