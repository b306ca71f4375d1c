"""The one-launch decode (fold_decode_fused) against the three calls and the oracle.

The fused call must give the bits of fold_ref_estimate + fold_decode_split +
fold_combine: Z, every slot of A and L, the output (fp32 or bf16), the base-2
log-sum-exp and the certificate.  Its output and Z are also held to the oracle
bars directly (row error <= 1e-2 |o_i|_inf at T = inf, |dZ| <= 1e-3 binades),
and its arrival counters must be zero after every call.
"""

import math

import numpy as np
import pytest
import torch

import paper_2609_33410_amd as F
from tests import _adapt, _gpu
from workloads import make_cascade, make_config, make_custom

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
    if t.dtype in (torch.float32, torch.int32):
        return t.view(torch.int32)
    if t.dtype in (torch.bfloat16, torch.int16):
        return t.view(torch.int16)
    return t


def _same(a, b, what):
    assert a.shape == b.shape, what
    ok = torch.equal(_bits(a), _bits(b))
    if not ok:
        d = (_bits(a) != _bits(b)).nonzero()
        print(f"  {what}: {d.shape[0]} elements differ, first at {d[0].tolist()}")
    assert ok, what


def _outputs(wl, splits, out_dtype):
    dev = wl.q.device
    b, h, d = wl.q.shape
    return {
        "part_A": torch.full((splits, b, h, d), NAN, dtype=torch.float32, device=dev),
        "part_L": torch.full((splits, b, h), NAN, dtype=torch.float32, device=dev),
        "z": torch.full((b, h), NAN, dtype=torch.float32, device=dev),
        "out": torch.full((b, h, d), NAN, dtype=out_dtype, device=dev),
        "lse": torch.full((b, h), NAN, dtype=torch.float32, device=dev),
        "cert": torch.full((b, h), 255, dtype=torch.uint8, device=dev),
    }


def fused(wl, T, splits, out_dtype=torch.float32, arrivals=None, params=None):
    (kv,), _ = _gpu.kv_views(wl)
    o = _outputs(wl, splits, out_dtype)
    if arrivals is None:
        arrivals = torch.zeros(wl.levels[0].num_seqs, wl.num_kv_heads, dtype=torch.int32,
                               device=wl.q.device)
    F.fold_decode_fused(kv, F.q_view(wl.q), wl.sm_scale, T, splits, o["part_A"], o["part_L"],
                        arrivals, o["z"], o["out"], lse_out=o["lse"], cert_out=o["cert"],
                        params=params)
    torch.cuda.synchronize()
    return {k: v.cpu() for k, v in o.items()}, arrivals


def three_calls(wl, T, splits, out_dtype=torch.float32, params=None):
    (kv,), flat = _gpu.kv_views(wl)
    qv = F.q_view(wl.q)
    o = _outputs(wl, splits, out_dtype)
    F.fold_ref_estimate(flat, qv, wl.sm_scale, o["z"], params=params)
    F.fold_decode_split(kv, qv, wl.sm_scale, o["z"], T, splits, 0, o["part_A"], o["part_L"])
    F.fold_combine(o["part_A"], o["part_L"], o["out"], z=o["z"], lse_out=o["lse"],
                   cert_out=o["cert"])
    torch.cuda.synchronize()
    return {k: v.cpu() for k, v in o.items()}


def check_same(wl, T, splits, out_dtype=torch.float32, params=None):
    print(f"  {wl.name} T={T} S={splits} out={out_dtype}", flush=True)
    got, arr = fused(wl, T, splits, out_dtype, params=params)
    ref = three_calls(wl, T, splits, out_dtype, params=params)
    for k in ("z", "part_A", "part_L", "out", "lse", "cert"):
        _same(got[k], ref[k], k)
    assert int(arr.abs().sum()) == 0, "arrival counters must be left at zero"
    return got


@pytest.mark.parametrize("splits", [1, 3, 8])
@pytest.mark.parametrize("T", [INF, 16.0, 4.0])
def test_fused_bits_config2_shape_small(splits, T):
    wl = make_config(2, batch=2, seq_len=1000, device="cuda")
    check_same(wl, T, splits)


def test_fused_bits_bf16_output():
    wl = make_config(2, batch=3, seq_len=777, device="cuda")
    for T in (INF, 16.0):
        check_same(wl, T, 4, out_dtype=torch.bfloat16)


@pytest.mark.parametrize("d", [64, 128])
@pytest.mark.parametrize("group", [2, 4, 8])
@pytest.mark.parametrize("paged", [True, False])
def test_fused_ragged_edge_lengths(d, group, paged):
    """Empty, single-key, page- and tile-boundary lengths; partial last tiles;
    the empty request's row gets the combine's NaN output and certificate."""
    lens = [0, 1, 15, 16, 17, 63, 64, 65, 200, 333]
    wl = make_custom(batch=len(lens), heads=2 * group, kv_heads=2, dim=d, lens=lens,
                     paged=paged, spike_count=2, n_sink=1, seed=d + group, device="cuda")
    for T, s in ((INF, 1), (6.0, 3), (16.0, 5)):
        got = check_same(wl, T, s)
        assert torch.isnan(got["out"][0]).all()
        assert ((got["cert"][0].numpy() & 5) == 5).all()


def test_fused_small_estimator_sample():
    """Custom estimator parameters with fewer sample tiles than waves (waves
    without a tile still issue their scan's first keys at the same point)."""
    params = {"sink": 4, "recent": 12, "strata": 8, "trim_lo": 1, "trim_hi": 1}
    wl = make_custom(batch=3, heads=16, kv_heads=2, dim=128, lens=[3000, 700, 90],
                     spike_count=6, n_sink=4, seed=21, device="cuda")
    for T in (INF, 16.0):
        check_same(wl, T, 2, params=params)


def test_fused_oracle_parity():
    """Z and the T = inf output of the fused call against the FP64 oracle."""
    wl = make_config(2, batch=2, seq_len=1000, device="cuda")
    oi = _adapt.oracle_inputs(wl)
    got, _ = fused(wl, INF, 3)
    zo = _adapt.estimate(oi)
    dz = np.abs(got["z"].double().numpy() - zo).max()
    print(f"  max |dZ| = {dz:.3e} binades")
    assert dz <= 1e-3
    o_ref, l_ref, _, _ = _adapt.decode(oi, got["z"].double().numpy(), INF, [3])
    err = _gpu.row_errors(got["out"].numpy(), o_ref)
    print(f"  max row err = {err.max():.3e}")
    assert (err <= 1e-2).all()
    lse_ref = got["z"].double().numpy() + np.log2(l_ref)
    assert np.abs(got["lse"].double().numpy() - lse_ref).max() <= 1e-4


def test_fused_consecutive_calls_share_arrivals():
    """Calls of different depth and split count in a row on one counter array:
    each gives the three calls' bits and leaves the counters at zero."""
    wl = make_config(2, batch=4, seq_len=1500, device="cuda")
    arrivals = torch.zeros(wl.levels[0].num_seqs, wl.num_kv_heads, dtype=torch.int32,
                           device="cuda")
    for T, s in ((INF, 4), (16.0, 1), (6.0, 7), (INF, 2)):
        got, arr = fused(wl, T, s, arrivals=arrivals)
        assert arr is arrivals
        assert int(arrivals.abs().sum()) == 0
        ref = three_calls(wl, T, s)
        for k in ("z", "out", "lse", "cert"):
            _same(got[k], ref[k], f"{k} T={T} S={s}")


@pytest.mark.parametrize("T", [INF, 16.0])
def test_fused_full_size_config2(T):
    """The Llama-3-8B-shaped workload at full size (16 x 8192 keys, paged), in
    the split count the benchmark times."""
    wl = make_config(2, device="cuda")
    check_same(wl, T, 4)


def test_fused_rejects_unsupported_shapes():
    def call(wl, out=None, splits=2, kv=None):
        levels, _ = _gpu.kv_views(wl)
        kv0 = levels[0]
        o = _outputs(wl, splits, torch.float32)
        arr = torch.zeros(max(wl.levels[0].num_seqs, 1), wl.num_kv_heads, dtype=torch.int32,
                          device="cuda")
        F.fold_decode_fused(kv if kv is not None else kv0, F.q_view(wl.q), wl.sm_scale, INF,
                            splits, o["part_A"], o["part_L"], arr, o["z"],
                            o["out"] if out is None else out)
        torch.cuda.synchronize()
        return o

    mha = make_custom(batch=2, heads=4, kv_heads=4, dim=64, lens=[100, 50], device="cuda")
    with pytest.raises(F.FoldError) as e:
        call(mha)
    assert e.value.status == F.FOLD_E_UNSUPPORTED
    g16 = make_custom(batch=2, heads=32, kv_heads=2, dim=64, lens=[100, 50], device="cuda")
    with pytest.raises(F.FoldError) as e:
        call(g16)
    assert e.value.status == F.FOLD_E_UNSUPPORTED
    wl = make_custom(batch=2, heads=8, kv_heads=2, dim=128, lens=[100, 50], device="cuda")
    b, h, d = wl.q.shape
    raw = torch.empty(b * h * d + 1, dtype=torch.float32, device="cuda")
    with pytest.raises(F.FoldError) as e:
        call(wl, out=raw[1:].view(b, h, d))
    assert e.value.status == F.FOLD_E_INVAL
    with pytest.raises(ValueError):  # fewer slots than splits: refused before the call
        F.fold_decode_fused(_gpu.kv_views(wl)[0][0], F.q_view(wl.q), wl.sm_scale, INF, 3,
                            torch.empty(2, b, h, d, device="cuda"),
                            torch.empty(2, b, h, device="cuda"),
                            torch.zeros(2, 2, dtype=torch.int32, device="cuda"),
                            torch.empty(b, h, device="cuda"), torch.empty(b, h, d, device="cuda"))
    casc = make_cascade(requests=3, heads=8, kv_heads=2, dim=128, prefix_len=128, suffix_len=32,
                        device="cuda")
    levels, _ = _gpu.kv_views(casc)
    with pytest.raises(F.FoldError) as e:
        call(casc, kv=levels[0])
    assert e.value.status == F.FOLD_E_INVAL
