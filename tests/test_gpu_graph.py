"""A whole per-tile step (pack x, unpack x, forward, pack dy, unpack dy,
weight gradient, input gradient: the path of Sec. III-A) captured once into
a HIP graph on a capture stream and replayed.  No entry point allocates,
frees, synchronizes or sets memory, so the capture holds only kernels; every
pass is deterministic, so each replay must reproduce the eager step bit for
bit.  Eager work runs between the replays.
"""
import pytest
import torch

import harness as H
import paper_1903_06681_amd as dc
from workloads import Layer
import workloads as wl

pytestmark = pytest.mark.gpu

X, DY, ALL = dc.DC_X, dc.DC_DY, dc.DC_ALL_TILES

# the centre tile of a 3x3 grid (all eight neighbours: every send region is
# written); 3x3 on whole 32-blocks and 128-column tiles, so the forward,
# input-gradient and k-slice weight-gradient kernels all run
LAYERS = [
    Layer("graph_bf16", 1, 32, 32, 384, 384, 3, 3, 1, 1, 3, 3, 1, "bf16", "uniform", 121),
    Layer("graph_f32", 2, 8, 16, 72, 48, 3, 3, 1, 1, 3, 3, 1, "f32", "uniform", 122),
]


def _bits(t):
    return t.view(torch.int16) if t.element_size() == 2 else t.view(torch.int32)


@pytest.mark.parametrize("L", LAYERS, ids=lambda L: L.name)
def test_graph_replay_reproduces_eager_step(L):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    p = dc.Problem.of(L)
    nt = L.P * L.Q
    tile = 4
    x, w, dy = wl.draw(L, "x"), wl.draw(L, "w"), wl.draw(L, "dy")
    tdt = H.TORCH_DT[L.dtype]
    xt = H.alloc_tiles(p, X, nt, L.dtype)
    H.scatter_interiors(xt, H.to_device(x, L.dtype), p, X)
    dyt = H.alloc_tiles(p, DY, nt, L.dtype)
    H.scatter_interiors(dyt, H.to_device(dy, L.dtype), p, DY)
    sx = torch.empty((nt, dc.halo_elems(p, X)), dtype=tdt, device="cuda")
    sy = torch.empty((nt, dc.halo_elems(p, DY)), dtype=tdt, device="cuda")
    dc.halo_pack(p, ALL, X, xt, sx)
    dc.halo_pack(p, ALL, DY, dyt, sy)
    recv_x, recv_dy = torch.zeros_like(sx[0]), torch.zeros_like(sy[0])
    H.exchange_into(recv_x, sx, p, X, tile)
    H.exchange_into(recv_dy, sy, p, DY, tile)
    xp, dyp = xt[tile].clone(), dyt[tile].clone()
    send_x, send_dy = torch.empty_like(recv_x), torch.empty_like(recv_dy)
    wd = H.to_device(w, L.dtype)
    y = torch.empty((L.N, L.K, L.Hot, L.Wot), device="cuda")
    dx = torch.empty((L.N, L.C, L.Ht, L.Wt), device="cuda")
    dw = torch.empty((L.K, L.C, L.R, L.S), device="cuda")
    ws = torch.empty(max(dc.bwd_filter_workspace_bytes(p, tile), 16), dtype=torch.uint8, device="cuda")

    def step(sp):
        dc.halo_pack(p, tile, X, xp, send_x, sp)
        dc.halo_unpack(p, tile, X, recv_x, xp, sp)
        dc.conv_fwd(p, tile, xp, wd, y, sp)
        dc.halo_pack(p, tile, DY, dyp, send_dy, sp)
        dc.halo_unpack(p, tile, DY, recv_dy, dyp, sp)
        dc.conv_bwd_filter(p, tile, xp, dyp, dw, 0, ws, sp)
        dc.conv_bwd_data(p, tile, dyp, wd, dx, sp)

    main = torch.cuda.current_stream()
    outs = (y, dx, dw, send_x, send_dy)
    for t in outs:
        t.fill_(float("nan"))
    step(main.cuda_stream)
    torch.cuda.synchronize()
    ref = [t.clone() for t in outs]
    assert all(bool(torch.isfinite(t.float()).all()) for t in ref)

    cap = torch.cuda.Stream()
    cap.wait_stream(main)
    with torch.cuda.stream(cap):
        step(cap.cuda_stream)
    main.wait_stream(cap)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=cap):
        step(cap.cuda_stream)
    torch.cuda.synchronize()

    for r in range(3):
        for t in outs:
            t.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        for name, a, b in zip(("y", "dx", "dw", "send_x", "send_dy"), outs, ref):
            assert torch.equal(_bits(a), _bits(b)), f"replay {r}: {name} differs from the eager step"
        step(main.cuda_stream)          # eager work between replays
        torch.cuda.synchronize()
        for a, b in zip(outs, ref):
            assert torch.equal(_bits(a), _bits(b))
