"""fold_decode_fused_noalloc (slots and arrival counts in the library's fixed
device scratch) against fold_decode_fused with caller workspace: the same
kernel, so Z, the output, the log-sum-exp and the certificate must agree bit
for bit (stricter than the 1e-2 row bar the oracle parity tests use).  Two
calls in a row, the second with a smaller input; a call too large for the
scratch is refused before anything launches."""

import math

import pytest
import torch

import paper_2609_33410_amd as F
from tests import _gpu
from workloads import make_config, make_custom

pytestmark = pytest.mark.gpu
INF = float("inf")
NAN = float("nan")


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    F.load_library()  # raises if the HIP library is not built: never a silent fallback


def _bits(t):
    t = t.contiguous()
    if t.dtype == torch.float32:
        return t.view(torch.int32)
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16)
    return t


def _outs(wl, out_dtype):
    b, h, d = wl.q.shape
    dev = wl.q.device
    return {"z": torch.full((b, h), NAN, device=dev),
            "out": torch.full((b, h, d), NAN, dtype=out_dtype, device=dev),
            "lse": torch.full((b, h), NAN, device=dev),
            "cert": torch.full((b, h), 255, dtype=torch.uint8, device=dev)}


def _with_workspace(wl, T, splits, out_dtype):
    (kv,), _ = _gpu.kv_views(wl)
    b, h, d = wl.q.shape
    dev = wl.q.device
    o = _outs(wl, out_dtype)
    pa = torch.full((splits, b, h, d), NAN, device=dev)
    pl = torch.full((splits, b, h), NAN, device=dev)
    arr = torch.zeros(wl.levels[0].num_seqs, wl.num_kv_heads, dtype=torch.int32, device=dev)
    F.fold_decode_fused(kv, F.q_view(wl.q), wl.sm_scale, T, splits, pa, pl, arr, o["z"],
                        o["out"], lse_out=o["lse"], cert_out=o["cert"])
    torch.cuda.synchronize()
    return {k: v.cpu() for k, v in o.items()}


def _no_alloc(wl, T, splits, out_dtype):
    (kv,), _ = _gpu.kv_views(wl)
    o = _outs(wl, out_dtype)
    F.fold_decode_fused_noalloc(kv, F.q_view(wl.q), wl.sm_scale, T, splits, o["z"], o["out"],
                                lse_out=o["lse"], cert_out=o["cert"])
    torch.cuda.synchronize()
    return {k: v.cpu() for k, v in o.items()}


def _same(a, b, what):
    for k in ("z", "out", "lse", "cert"):
        assert torch.equal(_bits(a[k]), _bits(b[k])), f"{what}: {k} differs"


@pytest.mark.parametrize("T", [INF, 16.0])
def test_no_alloc_matches_workspace_call_twice_then_smaller(T):
    """Two calls in a row on the scratch (the second smaller: fewer requests,
    shorter and ragged sequences, fewer splits, BF16 output), each bitwise
    equal to the workspace call on the same inputs; then the first input
    again, so leftovers of the small call change nothing."""
    big = make_config(2, batch=8, seq_len=4000, device="cuda")
    small = make_custom(batch=3, heads=16, kv_heads=4, dim=128, lens=[0, 333, 1500],
                        spike_count=4, n_sink=2, seed=5, device="cuda")
    for wl, splits, dt in ((big, 8, torch.float32), (small, 3, torch.bfloat16),
                           (big, 8, torch.float32)):
        ref = _with_workspace(wl, T, splits, dt)
        got = _no_alloc(wl, T, splits, dt)
        _same(got, ref, f"{wl.name} S={splits}")


def test_no_alloc_full_size_workload2():
    """The Llama-3-8B-shaped decode (16 requests x 8192 keys, 4 splits): its
    1 MiB of slots fit the scratch; bitwise equal to the workspace call."""
    wl = make_config(2, device="cuda")
    for T in (INF, 16.0):
        _same(_no_alloc(wl, T, 4, torch.float32), _with_workspace(wl, T, 4, torch.float32),
              f"workload 2 T={T}")


def test_no_alloc_refuses_calls_beyond_the_scratch():
    """64 splits x 16 requests x 32 heads x 129 floats = 16.9 MB > 8 MiB:
    refused with FOLD_E_INVAL before any launch; outputs untouched."""
    wl = make_config(2, batch=16, seq_len=256, device="cuda")
    (kv,), _ = _gpu.kv_views(wl)
    o = _outs(wl, torch.float32)
    with pytest.raises(F.FoldError) as ei:
        F.fold_decode_fused_noalloc(kv, F.q_view(wl.q), wl.sm_scale, INF, 64, o["z"], o["out"])
    assert ei.value.status == F.FOLD_E_INVAL
    assert "scratch" in str(ei.value)
    torch.cuda.synchronize()
    assert torch.isnan(o["out"]).all() and torch.isnan(o["z"]).all()
