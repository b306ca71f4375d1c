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
