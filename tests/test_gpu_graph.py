"""The whole decode step (estimate, split scans, combine) captured in one HIP
graph gives the eager result on every replay, with eager work in between."""

import math

import pytest
import torch

from tests import _gpu
from workloads import make_config

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


@pytest.mark.parametrize("cfg,T", [(2, math.inf), (2, 16.0), (5, 16.0), (4, math.inf)])
def test_graph_replays_match_eager(cfg, T):
    import paper_2609_33410_amd as F

    wl = make_config(cfg, device="cuda", batch=4 if cfg != 5 else 8,
                     seq_len=3000 if cfg != 4 else 5000)
    levels, flat = _gpu.kv_views(wl)
    qv = F.q_view(wl.q)
    b, h, d = wl.q.shape
    splits = wl.level_splits
    z = torch.empty(b, h, dtype=torch.float32, device="cuda")
    part_a = torch.empty(sum(splits), b, h, d, dtype=torch.float32, device="cuda")
    part_l = torch.empty(sum(splits), b, h, dtype=torch.float32, device="cuda")
    out = torch.empty(b, h, d, dtype=torch.float32, device="cuda")

    def step(stream):
        F.fold_ref_estimate(flat, qv, wl.sm_scale, z, stream=stream)
        off = 0
        for kv, s in zip(levels, splits):
            F.fold_decode_split(kv, qv, wl.sm_scale, z, T, s, off, part_a, part_l, stream=stream)
            off += s
        F.fold_combine(part_a, part_l, out, stream=stream)

    step(torch.cuda.current_stream())
    torch.cuda.synchronize()
    eager = out.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(torch.cuda.current_stream())
    for it in range(3):
        out.fill_(float("nan"))
        z.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager), f"replay {it} differs from the eager step"
        step(torch.cuda.current_stream())  # eager work between replays
        torch.cuda.synchronize()
        assert torch.equal(out, eager)


@pytest.mark.parametrize("T", [math.inf, 16.0])
def test_graph_replays_of_the_cascade_scan(T):
    """Estimate, the one-launch cascade scan and the combine captured in one
    graph: every replay gives the eager bits, with eager steps in between."""
    import paper_2609_33410_amd as F

    wl = make_config(5, device="cuda", batch=8, seq_len=3000)
    levels, flat = _gpu.kv_views(wl)
    qv = F.q_view(wl.q)
    b, h, d = wl.q.shape
    s = wl.level_splits[0]
    z = torch.empty(b, h, dtype=torch.float32, device="cuda")
    part_a = torch.empty(s, b, h, d, dtype=torch.float32, device="cuda")
    part_l = torch.empty(s, b, h, dtype=torch.float32, device="cuda")
    out = torch.empty(b, h, d, dtype=torch.float32, device="cuda")

    def step(stream):
        F.fold_ref_estimate(flat, qv, wl.sm_scale, z, stream=stream)
        F.fold_decode_cascade(levels[0], levels[1], qv, wl.sm_scale, z, T, s, 0, part_a, part_l,
                              stream=stream)
        F.fold_combine(part_a, part_l, out, stream=stream)

    step(torch.cuda.current_stream())
    torch.cuda.synchronize()
    eager = out.clone()
    assert torch.isfinite(eager).all()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(torch.cuda.current_stream())
    for it in range(3):
        out.fill_(float("nan"))
        part_a.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager), f"replay {it} differs from the eager step"
        step(torch.cuda.current_stream())
        torch.cuda.synchronize()
        assert torch.equal(out, eager)


@pytest.mark.parametrize("T", [math.inf, 16.0])
def test_graph_replays_of_the_fused_call(T):
    """The one-launch decode captured in a graph: every replay gives the eager
    bits and leaves the arrival counts at zero (they reset themselves, so the
    graph holds no memset), with eager calls on the same counters in between."""
    import paper_2609_33410_amd as F

    wl = make_config(2, device="cuda", batch=4, seq_len=3000)
    (kv,), _ = _gpu.kv_views(wl)
    qv = F.q_view(wl.q)
    b, h, d = wl.q.shape
    s = 4
    z = torch.empty(b, h, dtype=torch.float32, device="cuda")
    part_a = torch.empty(s, b, h, d, dtype=torch.float32, device="cuda")
    part_l = torch.empty(s, b, h, dtype=torch.float32, device="cuda")
    arrivals = torch.zeros(b, wl.num_kv_heads, dtype=torch.int32, device="cuda")
    out = torch.empty(b, h, d, dtype=torch.float32, device="cuda")
    lse = torch.empty(b, h, dtype=torch.float32, device="cuda")

    def call(stream):
        F.fold_decode_fused(kv, qv, wl.sm_scale, T, s, part_a, part_l, arrivals, z, out,
                            lse_out=lse, stream=stream)

    call(torch.cuda.current_stream())
    torch.cuda.synchronize()
    eager, eager_lse = out.clone(), lse.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call(torch.cuda.current_stream())
    for it in range(4):
        out.fill_(float("nan"))
        lse.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager), f"replay {it} differs from the eager call"
        assert torch.equal(lse, eager_lse)
        assert int(arrivals.abs().sum()) == 0
        call(torch.cuda.current_stream())  # eager work between replays
        torch.cuda.synchronize()
        assert torch.equal(out, eager)
