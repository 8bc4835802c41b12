"""Host tests of the per-layer performance model (Sec. V-A): its halo message
sizes against the library's packed regions, the communication closed forms,
the omission rules and the overlap combination (no GPU), and one GPU run of
the measurement that feeds it."""
import pytest

import harness as H
import paper_1903_06681_amd as dc
from paper_1903_06681_amd import perfmodel as pm

LAYERS = [
    pm.LayerShape(4, 64, 64, 1024, 1024, 3, 3, 1, 1, 1, "bf16"),
    pm.LayerShape(2, 32, 48, 72, 96, 5, 5, 1, 2, 2, "bf16"),
    pm.LayerShape(1, 18, 32, 2048, 2048, 3, 3, 1, 1, 1, "f32"),
    pm.LayerShape(8, 3, 64, 224, 224, 7, 7, 2, 3, 3, "bf16"),
]


def _prob(layer, d):
    return dc.Problem(layer.N // d.s, layer.C, layer.F, layer.H, layer.W, layer.R, layer.S,
                      layer.stride, layer.pad, d.P, d.Q, layer.halo,
                      dc.DC_BF16 if layer.dtype == "bf16" else dc.DC_F32)


@pytest.mark.parametrize("layer", LAYERS)
@pytest.mark.parametrize("grid", [(1, 2), (2, 1), (2, 2), (4, 4), (2, 4)])
@pytest.mark.parametrize("which", ["x", "dy"])
def test_halo_messages_match_library_regions(layer, grid, which):
    """Every message of Sec. V-A equals the library's packed send region for
    that direction (elements), and regions without a neighbour carry none."""
    d = pm.Distribution(1, *grid)
    if d not in pm.candidate_distributions(layer, d.gpus):
        pytest.skip("not a valid split of this layer")
    prob = _prob(layer, d)
    assert dc.validate(prob, (d.P // 2) * d.Q + d.Q // 2) == 0
    w = dc.DC_X if which == "x" else dc.DC_DY
    table = H.region_table(prob, w, send=True)
    assert pm.halo_bands(layer, d, which) == dc.halo_bands(prob, w)
    ch = layer.C if which == "x" else layer.F
    msgs = dict(pm.halo_messages(layer, d, which))
    for direction, (_, rows, cols) in table.items():
        di, dj = H.STEP[direction]
        present = (di == 0 or d.P > 1) and (dj == 0 or d.Q > 1)
        if present:
            assert msgs[direction] == prob.N * ch * rows * cols, direction
        else:
            assert direction not in msgs
    if d.P > 1 and d.Q > 1:
        al = 8 if layer.dtype == "bf16" else 4   # packed buffers end on a 16-byte boundary
        assert -(-sum(msgs.values()) // al) * al == dc.halo_elems(prob, w)


def test_no_messages_without_spatial_split():
    layer = LAYERS[0]
    assert pm.halo_messages(layer, pm.Distribution(4, 1, 1), "x") == []
    assert pm.halo_messages(layer, pm.Distribution(4, 1, 1), "dy") == []


def test_paper_message_sizes_written_out():
    """Sec. V-A for a P x Q split: 2 x O*n*c*w (north/south), 2 x O*n*c*h
    (east/west), 4 x O^2*n*c (corners)."""
    layer = pm.LayerShape(8, 16, 24, 64, 96, 3, 3, 1, 1, 1, "bf16")
    d = pm.Distribution(2, 2, 3)
    n, h, w = 4, 32, 32
    O, c = 1, 16
    m = pm.halo_messages(layer, d, "x")
    assert sorted(v for _, v in m) == sorted([O * n * c * w] * 2 + [O * n * c * h] * 2 + [O * O * n * c] * 4)


def test_link_and_allreduce_closed_forms():
    link = pm.Link(alpha=2e-6, beta=1e-9)
    assert link.sr(0) == 0.0
    assert link.sr(1000) == pytest.approx(2e-6 + 1e-6)
    assert pm.allreduce_time(1, 1e6, link) == 0.0
    # p = 2: recursive doubling is one exchange: alpha + n beta
    assert pm.allreduce_time(2, 1e6, link) == pytest.approx(2e-6 + 1e-3)
    # large n, p = 8: the ring's 2(p-1)/p n beta beats log2(p) n beta
    n = 1e9
    ring = 14 * 2e-6 + 1.75 * n * 1e-9
    assert pm.allreduce_time(8, n, link) == pytest.approx(ring)
    # small n, p = 8: three latency terms of recursive doubling beat 14 of the ring
    assert pm.allreduce_time(8, 8, link) == pytest.approx(3 * (2e-6 + 8e-9))


def test_exchange_serial_is_sum_concurrent_is_max():
    link = pm.Link(1e-6, 1e-9)
    msgs = [("N", 100), ("S", 100), ("W", 300), ("E", 300)]
    assert pm.exchange_time(msgs, 2, link, concurrent=False) == pytest.approx(4e-6 + 1600e-9)
    assert pm.exchange_time(msgs, 2, link, concurrent=True) == pytest.approx(1e-6 + 600e-9)


def test_candidates_are_balanced_and_valid():
    layer = LAYERS[0]
    for g in (1, 2, 4, 8, 16):
        for d in pm.candidate_distributions(layer, g):
            assert d.gpus == g and layer.N % d.s == 0
            assert dc.validate(_prob(layer, d), 0) == 0
    # N = 4: at most 4 sample groups
    assert all(d.s <= 4 for d in pm.candidate_distributions(layer, 16))
    assert pm.Distribution(4, 2, 2) in pm.candidate_distributions(layer, 16)
    assert pm.Distribution(1, 4, 4) in pm.candidate_distributions(layer, 16)


def test_overlapped_never_slower_and_sample_parallelism_is_cheapest():
    """With compute split perfectly, a spatial split only adds halo terms:
    sample parallelism has the least communication (Sec. V-A)."""
    layer = pm.LayerShape(8, 64, 64, 256, 256, 3, 3, 1, 1, 1, "bf16")
    link = pm.xgmi_link()
    base = pm.TileTimes(C=80e-6, Cx=80e-6, Cw=90e-6)
    times = {}
    for d in pm.candidate_distributions(layer, 4):
        k = d.gpus
        times[d] = pm.TileTimes(C=base.C / k, Cx=base.Cx / k, Cw=base.Cw / k,
                                pack_x=3e-6, unpack_x=3e-6, pack_dy=3e-6, unpack_dy=3e-6)
    for mode in ("serial", "overlapped"):
        preds = pm.best_distribution(layer, 4, times, link, mode)
        assert preds[0].dist == pm.Distribution(4, 1, 1)
    for d, t in times.items():
        s = pm.predict(layer, d, t, link, "serial")
        o = pm.predict(layer, d, t, link, "overlapped")
        assert o.total <= s.total + 1e-15
        assert s.total == pytest.approx(s.FP + s.BPx + s.BPw + s.BPa)
    # a 2 x 2 split pays two exchanges of eight messages each
    d = pm.Distribution(1, 2, 2)
    p = pm.predict(layer, d, times[d], link, "serial", concurrent_links=False)
    assert p.halo_x > 8 * link.alpha and p.halo_dy > 8 * link.alpha


@pytest.mark.gpu
def test_measured_times_feed_the_model():
    """measure_tile times the five calls on one tile of each split; the
    model then ranks the splits (small layer, a few milliseconds of GPU work)."""
    layer = pm.LayerShape(4, 32, 32, 64, 64, 3, 3, 1, 1, 1, "bf16")
    times = {d: pm.measure_tile(layer, d, reps=3, warmup=1) for d in pm.candidate_distributions(layer, 4)}
    for d, t in times.items():
        assert t.C > 0 and t.Cx > 0 and t.Cw > 0
        if d.P * d.Q > 1:
            assert min(t.pack_x, t.unpack_x, t.pack_dy, t.unpack_dy) > 0
    preds = pm.best_distribution(layer, 4, times, pm.xgmi_link())
    assert len(preds) == len(times) and preds[0].total <= preds[-1].total
