"""Per-layer performance model for sample + spatial parallelism (Sec. V-A).

The paper estimates a convolutional layer's time under a distribution from
*measured* local convolution times and an *analytic* communication model:

  FP  = C(n, c, h, w, f)  + halo exchange of x  (Sec. V-A)
  BPx = Cx(n, c, h, w, f) + halo exchange of dL/dy
  BPw = Cw(n, c, h, w, f)
  BPa = AR(p, f * c * K^2)                      (allreduce of dL/dw)

with lower-case shapes local to one GPU.  A halo exchange with margin width
O sends two north/south messages of O*n*ch*w elements, two east/west ones of
O*n*ch*h and four corners of O^2*n*ch (with stride > 1 each side carries
the band its receiver reads, which may be narrower); the east/west and corner
messages vanish when the width is not split, the north/south and corner ones
when the height is not split.  Point-to-point messages follow the linear model
SR(m) = alpha + beta*m (full duplex, no interference, Sec. II-B); allreduces
follow the collective models the paper cites (ring / recursive doubling).

Here C, Cx, Cw are the times of this library's kernels on one tile
(dc_conv_fwd, dc_conv_bwd_data, dc_conv_bwd_filter), and the local halo work
(dc_halo_pack, dc_halo_unpack) is measured too; only the wire time is
analytic, since one GPU cannot measure it.  Two ways to combine the terms:

* ``serial``: the paper's sums, nothing overlapped;
* ``overlapped``: the overlaps the paper lists that this implementation can
  realise -- the dL/dy exchange runs beside dL/dw, the allreduce beside dL/dx.

``best_distribution`` enumerates the sample x P x Q splits of a layer over G
GPUs and ranks them by predicted time per layer and step.

The model part is plain Python; ``measure_tile`` times the kernels on the
current GPU (it needs torch and a built library).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, Iterable, List, Optional, Tuple

ELEM_BYTES = {"f32": 4, "bf16": 2}
# y, dx, dw and partial sums are fp32; dL/dw travels in fp32
GRAD_BYTES = 4


@dataclasses.dataclass(frozen=True)
class Link:
    """Linear point-to-point cost SR(m) = alpha + beta * m (seconds, bytes)."""
    alpha: float
    beta: float

    def sr(self, nbytes: float) -> float:
        return 0.0 if nbytes <= 0 else self.alpha + self.beta * nbytes


def xgmi_link(gbytes_per_s: float = 153.6, latency_s: float = 10e-6) -> Link:
    """An assumed MI355X peer link: one neighbour per point-to-point xGMI link.

    Neither figure is measured here (one GPU): the bandwidth is the public
    per-link rate, the latency a typical small-message send/recv; both are
    parameters of the model.
    """
    return Link(alpha=latency_s, beta=1.0 / (gbytes_per_s * 1e9))


def allreduce_time(p: int, nbytes: float, link: Link) -> float:
    """AR(p, n): the cheaper of ring (reduce-scatter + allgather) and
    recursive doubling, the two regimes of the collective models the paper
    uses.  Reduction arithmetic is not counted."""
    if p <= 1 or nbytes <= 0:
        return 0.0
    ring = 2 * (p - 1) * link.alpha + 2.0 * (p - 1) / p * nbytes * link.beta
    rd = math.ceil(math.log2(p)) * (link.alpha + nbytes * link.beta)
    return min(ring, rd)


@dataclasses.dataclass(frozen=True)
class LayerShape:
    """A convolutional layer (paper notation: N samples, C channels, H x W,
    F filters of K x K) with this library's stride / padding / margin."""
    N: int
    C: int
    F: int
    H: int
    W: int
    R: int
    S: int
    stride: int = 1
    pad: int = 0
    halo: int = 0          # margin width O on every side of a tile
    dtype: str = "bf16"

    @property
    def Ho(self) -> int:
        return (self.H + 2 * self.pad - self.R) // self.stride + 1

    @property
    def Wo(self) -> int:
        return (self.W + 2 * self.pad - self.S) // self.stride + 1


@dataclasses.dataclass(frozen=True)
class Distribution:
    """s sample groups x a P x Q spatial grid: s * P * Q GPUs."""
    s: int
    P: int
    Q: int

    @property
    def gpus(self) -> int:
        return self.s * self.P * self.Q


def local_dims(layer: LayerShape, d: Distribution) -> Tuple[int, int, int, int, int]:
    """(n, h, w, ho, wo): samples, input and output tile extents on one GPU."""
    n = layer.N // d.s
    if d.P == 1 and d.Q == 1:
        return n, layer.H, layer.W, layer.Ho, layer.Wo
    h, w = layer.H // d.P, layer.W // d.Q
    return n, h, w, h // layer.stride, w // layer.stride


def halo_bands(layer: LayerShape, d: Distribution, which: str) -> Tuple[int, int, int, int]:
    """Band widths (above, below, left, right) of a tile's x halo ('x': the
    rows and columns Eq. (1) reads beyond the tile) or dL/dy halo ('dy':
    Eq. (3)).  At stride 1 with 'same' padding all four are O = layer.halo's
    usual value; at stride > 1 one side may need fewer (Sec. III-A)."""
    _, h, w, ho, wo = local_dims(layer, d)

    def x_side(t_in, t_out, R):
        return layer.pad, max(0, (t_out - 1) * layer.stride - layer.pad + R - 1 - (t_in - 1))

    def dy_side(t_in, t_out, R):
        st = layer.stride
        mmin = -((R - 1 - layer.pad) // st)          # ceil((pad - (R-1)) / stride)
        mmax = (t_in - 1 + layer.pad) // st
        return max(0, -mmin), max(0, mmax - (t_out - 1))

    side = x_side if which == "x" else dy_side
    a, b = side(h, ho, layer.R)
    l, r = side(w, wo, layer.S)
    return a, b, l, r


def halo_messages(layer: LayerShape, d: Distribution, which: str) -> List[Tuple[str, int]]:
    """Messages one interior GPU sends for the x halo ('x', forward) or the
    dL/dy halo ('dy', backward-data): (direction, elements), following the
    region list of Sec. V-A.  A message toward direction d carries the band
    the neighbour there reads on its opposite side (margin width O on every
    side for the stride-1 layers of the paper)."""
    n, h, w, ho, wo = local_dims(layer, d)
    if layer.halo == 0 or (d.P == 1 and d.Q == 1):
        return []
    ch, th, tw = (layer.C, h, w) if which == "x" else (layer.F, ho, wo)
    bn, bs, bw, be = halo_bands(layer, d, which)
    msgs = []
    if d.P > 1:
        msgs += [("N", bs * n * ch * tw), ("S", bn * n * ch * tw)]
    if d.Q > 1:
        msgs += [("W", be * n * ch * th), ("E", bw * n * ch * th)]
    if d.P > 1 and d.Q > 1:
        msgs += [("NW", bs * be * n * ch), ("NE", bs * bw * n * ch),
                 ("SW", bn * be * n * ch), ("SE", bn * bw * n * ch)]
    return msgs


def exchange_time(msgs: Iterable[Tuple[str, int]], elem_bytes: int, link: Link,
                  concurrent: bool) -> float:
    """Wire time of one halo exchange: the paper's sum of SR terms, or (one
    neighbour per link, all links at once) the slowest message."""
    t = [link.sr(m * elem_bytes) for _, m in msgs]
    if not t:
        return 0.0
    return max(t) if concurrent else sum(t)


@dataclasses.dataclass
class TileTimes:
    """Measured local times of one tile (seconds)."""
    C: float        # forward
    Cx: float       # backward-data
    Cw: float       # backward-filter (local dL/dw, including its reduction)
    pack_x: float = 0.0
    unpack_x: float = 0.0
    pack_dy: float = 0.0
    unpack_dy: float = 0.0


@dataclasses.dataclass
class Prediction:
    dist: Distribution
    FP: float
    BPx: float
    BPw: float
    BPa: float
    total: float
    halo_x: float
    halo_dy: float


def predict(layer: LayerShape, d: Distribution, t: TileTimes, link: Link,
            mode: str = "overlapped", concurrent_links: bool = True) -> Prediction:
    """Time of one layer (forward + backward) on each GPU under distribution d.

    serial:     FP + BPx + BPw + BPa as in Sec. V-A;
    overlapped: the dL/dy exchange hides behind BPw and the allreduce behind
                BPx (two of the overlaps Sec. V-A lists); the forward halo
                is not overlapped (no interior/boundary split here)."""
    eb = ELEM_BYTES[layer.dtype]
    wire_x = exchange_time(halo_messages(layer, d, "x"), eb, link, concurrent_links)
    wire_dy = exchange_time(halo_messages(layer, d, "dy"), eb, link, concurrent_links)
    spatial = d.P * d.Q > 1
    halo_x = (t.pack_x + wire_x + t.unpack_x) if spatial else 0.0
    halo_dy = (t.pack_dy + wire_dy + t.unpack_dy) if spatial else 0.0
    FP = t.C + halo_x
    BPx = t.Cx + halo_dy
    BPw = t.Cw
    BPa = allreduce_time(d.gpus, layer.F * layer.C * layer.R * layer.S * GRAD_BYTES, link)
    if mode == "serial":
        total = FP + BPx + BPw + BPa
    elif mode == "overlapped":
        total = FP + max(BPw, halo_dy) + t.Cx + max(0.0, BPa - t.Cx)
    else:
        raise ValueError(mode)
    return Prediction(d, FP, BPx, BPw, BPa, total, halo_x, halo_dy)


def candidate_distributions(layer: LayerShape, gpus: int) -> List[Distribution]:
    """Load-balanced splits s * P * Q = gpus: s divides N, P and Q divide H
    and W, decomposed tiles keep whole output tiles (stride) and are at least
    the margin wide."""
    out = []
    for s in range(1, gpus + 1):
        if gpus % s or layer.N % s:
            continue
        pq = gpus // s
        for P in range(1, pq + 1):
            if pq % P:
                continue
            Q = pq // P
            if P * Q == 1:
                out.append(Distribution(s, 1, 1))
                continue
            if layer.H % P or layer.W % Q:
                continue
            h, w = layer.H // P, layer.W // Q
            if h % layer.stride or w % layer.stride:
                continue
            if layer.Ho * layer.stride != layer.H or layer.Wo * layer.stride != layer.W:
                continue
            if (P > 1 and h < layer.halo) or (Q > 1 and w < layer.halo):
                continue
            out.append(Distribution(s, P, Q))
    return out


def best_distribution(layer: LayerShape, gpus: int, times: Dict[Distribution, TileTimes],
                      link: Link, mode: str = "overlapped") -> List[Prediction]:
    """Predictions for every candidate with measured times, fastest first."""
    preds = [predict(layer, d, times[d], link, mode) for d in candidate_distributions(layer, gpus)
             if d in times]
    return sorted(preds, key=lambda p: p.total)


# ---------------------------------------------------------------- measurement (GPU)

def measure_tile(layer: LayerShape, d: Distribution, reps: int = 20, warmup: int = 3) -> TileTimes:
    """Times this library's five calls on one tile of distribution d on the
    current GPU: K back-to-back launches between two events on the launch
    stream, averaged.  The tile is an interior one when the grid has one."""
    import torch
    import paper_1903_06681_amd as dc

    n = layer.N // d.s
    prob = dc.Problem(n, layer.C, layer.F, layer.H, layer.W, layer.R, layer.S, layer.stride,
                      layer.pad, d.P, d.Q, layer.halo,
                      dc.DC_BF16 if layer.dtype == "bf16" else dc.DC_F32)
    tile = (d.P // 2) * d.Q + d.Q // 2
    st = dc.validate(prob, tile)
    if st != 0:
        raise dc.DcError(st, f"measure_tile {d}")
    tdt = torch.bfloat16 if layer.dtype == "bf16" else torch.float32
    Ht, Wt, Hot, Wot = dc.tile_dims(prob)
    xp = torch.full(dc.tile_shape(prob, dc.DC_X), 0.5, dtype=tdt, device="cuda")
    dyp = torch.full(dc.tile_shape(prob, dc.DC_DY), 0.25, dtype=tdt, device="cuda")
    w = torch.full((layer.F, layer.C, layer.R, layer.S), 0.125, dtype=tdt, device="cuda")
    y = torch.empty((n, layer.F, Hot, Wot), device="cuda")
    dx = torch.empty((n, layer.C, Ht, Wt), device="cuda")
    dw = torch.empty((layer.F, layer.C, layer.R, layer.S), device="cuda")
    ws = torch.empty(max(dc.bwd_filter_workspace_bytes(prob, tile), 16), dtype=torch.uint8,
                     device="cuda")
    hx = max(dc.halo_elems(prob, dc.DC_X), 1)
    hdy = max(dc.halo_elems(prob, dc.DC_DY), 1)
    sx, rx = (torch.zeros(hx, dtype=tdt, device="cuda") for _ in range(2))
    sdy, rdy = (torch.zeros(hdy, dtype=tdt, device="cuda") for _ in range(2))
    calls = {
        "C": lambda: dc.conv_fwd(prob, tile, xp, w, y),
        "Cx": lambda: dc.conv_bwd_data(prob, tile, dyp, w, dx),
        "Cw": lambda: dc.conv_bwd_filter(prob, tile, xp, dyp, dw, 0, ws),
    }
    if d.P * d.Q > 1:
        calls.update({
            "pack_x": lambda: dc.halo_pack(prob, tile, dc.DC_X, xp, sx),
            "unpack_x": lambda: dc.halo_unpack(prob, tile, dc.DC_X, rx, xp),
            "pack_dy": lambda: dc.halo_pack(prob, tile, dc.DC_DY, dyp, sdy),
            "unpack_dy": lambda: dc.halo_unpack(prob, tile, dc.DC_DY, rdy, dyp),
        })
    out = {}
    stream = torch.cuda.current_stream()
    for k, f in calls.items():
        for _ in range(warmup):
            f()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(reps):
            f()
        e1.record(stream)
        torch.cuda.synchronize()
        out[k] = e0.elapsed_time(e1) / reps * 1e-3
    return TileTimes(**out)


def format_table(layer: LayerShape, gpus: int, preds: List[Prediction],
                 times: Dict[Distribution, TileTimes]) -> str:
    us = 1e6
    lines = [f"G={gpus}: {'s x P x Q':>10s} {'C':>8s} {'Cx':>8s} {'Cw':>8s} {'halo x':>8s} "
             f"{'halo dy':>8s} {'BPa':>8s} {'total':>9s}  (us)"]
    for i, p in enumerate(preds):
        t = times[p.dist]
        d = p.dist
        lines.append(f"{'best' if i == 0 else '':>4s}   {d.s:>3d} x {d.P} x {d.Q}   {t.C * us:8.1f} "
                     f"{t.Cx * us:8.1f} {t.Cw * us:8.1f} {p.halo_x * us:8.1f} {p.halo_dy * us:8.1f} "
                     f"{p.BPa * us:8.1f} {p.total * us:9.1f}")
    return "\n".join(lines)


def source_digest() -> str:
    """sha256 over the library's kernel and host sources (the timings belong to them)."""
    import hashlib
    import os

    d = os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc")
    h = hashlib.sha256()
    for f in sorted(os.listdir(d)):
        if f.endswith((".hip", ".h", ".cpp")):
            h.update(f.encode())
            with open(os.path.join(d, f), "rb") as fh:
                h.update(fh.read())
    return h.hexdigest()


def main(argv: Optional[List[str]] = None) -> None:
    """python -m paper_1903_06681_amd.perfmodel: measure and rank the splits
    of a few layers on the current GPU."""
    import argparse

    ap = argparse.ArgumentParser(description=main.__doc__)
    ap.add_argument("--gpus", type=int, nargs="+", default=[1, 2, 4, 8, 16])
    ap.add_argument("--mode", default="overlapped", choices=["overlapped", "serial"])
    ap.add_argument("--link-gbps", type=float, default=153.6)
    ap.add_argument("--latency-us", type=float, default=10.0)
    args = ap.parse_args(argv)
    link = xgmi_link(args.link_gbps, args.latency_us * 1e-6)
    print(f"source_sha256: {source_digest()}", flush=True)
    layers = {
        # ResNet-50 stage-2 3x3 layer, mini-batch 32 (Sec. VI-A microbenchmarks)
        "3x3 64->64 56x56, N=32": LayerShape(32, 64, 64, 56, 56, 3, 3, 1, 1, 1, "bf16"),
        # large-sample layer: 3x3 64->64 on 1024x1024, mini-batch 32
        "3x3 64->64 1024x1024, N=32": LayerShape(32, 64, 64, 1024, 1024, 3, 3, 1, 1, 1, "bf16"),
        # the same layer with 4 samples: its 1 x 4 x 4 split is the benchmark's tile
        "3x3 64->64 1024x1024, N=4": LayerShape(4, 64, 64, 1024, 1024, 3, 3, 1, 1, 1, "bf16"),
        # mesh-model first layer: 18 -> 32 channels on 2048x2048 fp32, one sample per step
        "3x3 18->32 2048x2048 fp32, N=1": LayerShape(1, 18, 32, 2048, 2048, 3, 3, 1, 1, 1, "f32"),
    }
    for name, layer in layers.items():
        print(f"== {name} (link {args.link_gbps} GB/s, alpha {args.latency_us} us, {args.mode})",
              flush=True)
        import paper_1903_06681_amd as dc
        cache: Dict[Distribution, TileTimes] = {}
        for g in args.gpus:
            skipped = []
            for d in candidate_distributions(layer, g):
                if d not in cache and d not in skipped:
                    try:
                        cache[d] = measure_tile(layer, d)
                    except dc.DcError as e:   # e.g. a tile past 32-bit element indexing
                        skipped.append(d)
                        print(f"   {d.s} x {d.P} x {d.Q}: not run ({e})", flush=True)
            preds = best_distribution(layer, g, cache, link, args.mode)
            print(format_table(layer, g, preds, cache), flush=True)


if __name__ == "__main__":
    main()
