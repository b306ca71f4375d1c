"""Parity of the stacked level over a two-plane key cache (Appendix E, tile
layouts: past 64 stacked rows one FP16 product per logit of each key's code,
rounded once per prefix) on the GPU.

Bars: the FP16 keys bit-exact against the oracle's rounding of the GPU's own
planes (byte work); the read bits of every 64-row read group bit-exact
against the FP32 rule on the exported x; the exported x equal to the
oracle's eta (k^ . q^) - Z to 1e-5 relative; per-slot L to 2e-5; outputs
within 1e-2 of the row's inf-norm in imposed mode (the decode's bar); the
production kernel's slots bitwise equal to the debug variant's.
"""

import math

import numpy as np
import pytest
import torch

import oracle
import paper_2609_33410_amd as F
from oracle import q8_oracle as q8
from tests import _adapt, _gpu, _gpu_q8
from workloads import host_bits, make_cascade

pytestmark = pytest.mark.gpu
INF = float("inf")
TOL = 1e-2


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    F.load_library()


def _stacked_view(wl, keys, k16, lv):
    return F.kv_view(k16, wl.v, lv.seq_lens, num_kv_heads=wl.num_kv_heads,
                     max_seq_len=lv.max_seq_len, block_table=lv.block_table,
                     row_indptr=lv.row_indptr, row_req=lv.row_req,
                     max_reqs_per_seq=lv.max_reqs_per_seq)


def _stack(wl, keys, lv):
    """FP16 keys of a level's sequences (NaN bits elsewhere)."""
    k16 = torch.full(keys.plane_a.shape, float("nan"), dtype=torch.float16, device=wl.k.device)
    layout = F.kv_view(keys.plane_a, None, lv.seq_lens, num_kv_heads=wl.num_kv_heads,
                       max_seq_len=lv.max_seq_len, block_table=lv.block_table,
                       row_indptr=lv.row_indptr, row_req=lv.row_req,
                       max_reqs_per_seq=lv.max_reqs_per_seq, k_is_layout_only=True)
    F.fold_q8_stack_keys(layout, keys, k16)
    return k16


CASES = {
    "40rows": dict(requests=5, heads=8, kv_heads=1, dim=128, prefix_len=1488, suffix_len=48,
                   splits=(3, 2)),
    "72rows_2kv": dict(requests=9, heads=16, kv_heads=2, dim=128, prefix_len=400,
                       suffix_len=32, splits=(2, 1)),
    "64rows_d64": dict(requests=8, heads=8, kv_heads=1, dim=64, prefix_len=720, suffix_len=16,
                       splits=(4, 1)),
}


def test_stacked_keys_bit_exact():
    wl = make_cascade(seed=1, device="cuda", **CASES["40rows"])
    keys = _gpu_q8.encode_cache(wl)
    k16 = _stack(wl, keys, wl.levels[0])
    torch.cuda.synchronize()
    a, b, e = (keys.plane_a.cpu().numpy(), keys.plane_b.cpu().numpy(),
               keys.scale.cpu().numpy().view(np.uint16))
    want = q8.stack_keys(a, b, e).view(np.uint16)
    got = k16.cpu().numpy().view(np.uint16)
    lv = wl.levels[0]
    bt = lv.block_table.cpu().numpy()
    n = lv.seq_lens_host[0]
    pages = bt[0, :(n + 15) // 16]
    assert np.array_equal(got[pages], want[pages])  # the prefix's pages, every element
    # pages of other sequences are not written
    others = np.setdiff1d(np.arange(got.shape[0]), pages)
    assert torch.isnan(k16.cpu()[torch.from_numpy(others)].float()).all()


@pytest.mark.parametrize("case", list(CASES))
@pytest.mark.parametrize("T", [INF, 16.0, 6.0])
def test_stacked_level_parity(case, T):
    """The prefix level (40, 72 or 64 stacked rows) on the FP16 keys against the
    oracle; then the whole cascade, the suffix on the two-plane gated scan."""
    wl = make_cascade(seed=2, device="cuda", **CASES[case])
    dev = wl.q.device
    keys = _gpu_q8.encode_cache(wl)
    qq = _gpu_q8.split_query(wl, 0.0)
    z = _gpu_q8.estimate(wl, keys, qq)
    levels, _ = _gpu_q8.level_views(wl, keys)
    lv0 = wl.levels[0]
    k16 = _stack(wl, keys, lv0)
    kv0 = _stacked_view(wl, keys, k16, lv0)
    assert F.fold_decode_rows_per_group(kv0, F.q_view(wl.q)) == 64
    b, h, d = wl.q.shape
    s0, s1 = wl.level_splits
    pa = torch.full((s0 + s1, b, h, d), float("nan"), device=dev)
    pl = torch.full((s0 + s1, b, h), float("nan"), device=dev)
    pa_d, pl_d = pa.clone(), pl.clone()
    rg = F.fold_decode_row_groups(kv0, F.q_view(wl.q))
    x = torch.full((b, h, lv0.max_seq_len), float("nan"), device=dev)
    kg = torch.full((1, wl.num_kv_heads, rg, lv0.max_seq_len), 255, dtype=torch.uint8, device=dev)
    F.fold_q8_decode_stacked(kv0, qq, z, T, s0, 0, pa, pl)
    F.fold_q8_decode_stacked(kv0, qq, z, T, s0, 0, pa_d, pl_d, x_out=x, key_gate_out=kg)
    F.fold_q8_decode_split(levels[1], keys, qq, z, T, s1, s0, pa, pl)
    out = torch.empty(b, h, d, device=dev)
    F.fold_combine(pa, pl, out)
    torch.cuda.synchronize()
    assert torch.equal(pa[:s0], pa_d[:s0]) and torch.equal(pl[:s0], pl_d[:s0])

    oi = _adapt.oracle_inputs(wl)
    a_, b_, e_ = (keys.plane_a.cpu().numpy(), keys.plane_b.cpu().numpy(),
                  keys.scale.cpu().numpy().view(np.uint16))
    khat = q8.stack_keys(a_, b_, e_)
    planes = qq.planes.cpu().numpy()
    qa, qb = planes[:, :, 0], planes[:, :, 1]
    qhat = q8.stack_queries(qa, qb)
    eta = qq.eta.cpu().numpy()
    z64 = z.cpu().double().numpy()
    lvo = oi["levels"][0]
    xg = x.cpu().numpy()
    # exported x against the oracle's logits; read bits against the FP32 rule
    G = wl.group
    n = lvo["seq_lens"][0]
    reqs = list(lvo["row_req"][lvo["row_indptr"][0]:lvo["row_indptr"][1]])
    for g in range(wl.num_kv_heads):
        kk = q8._gather_raw(khat, 0, g, n, lvo["block_table"], wl.page_size).astype(np.float64)
        rows = [(r, g * G + hh) for r in reqs for hh in range(G)]
        worst = 0.0
        for r, hh in rows:
            s = float(eta[r, hh]) * (kk @ qhat[r, hh].astype(np.float64))
            ref = s - z64[r, hh]
            worst = max(worst, float((np.abs(xg[r, hh, :n] - ref) / np.maximum(1.0, np.abs(s))).max()))
        assert worst <= 1e-5, worst
        for u in range(rg):
            grp = rows[64 * u:64 * (u + 1)]
            if not grp:
                continue
            live = np.stack([oracle.live_mask_imposed(xg[r, hh, :n], T) for r, hh in grp])
            vkey, _ = oracle.read_gates(live, n)
            assert np.array_equal(kg[0, g, u, :n].cpu().numpy().astype(bool), vkey), (g, u)
    a0, l0 = q8.decode_level_q8_stacked(qhat, eta, khat, oi["v_bits"],
                                        num_kv_heads=wl.num_kv_heads, page_size=wl.page_size,
                                        z=z64, T=T, num_splits=s0, imposed_x=xg, **lvo)
    tau = qq.tau.cpu().numpy()
    # the suffix level's decisions in the oracle's own FP64 (its parity is the
    # two-plane scan's, tested elsewhere); the bar covers both
    a1, l1 = q8.decode_level_q8(qa, qb, eta, (a_, b_, e_), oi["v_bits"],
                                num_kv_heads=wl.num_kv_heads, page_size=wl.page_size, z=z64,
                                T=T, tau=tau, num_splits=s1, **oi["levels"][1])
    gl = pl.cpu().double().numpy()
    cov = l0 > 0
    assert np.allclose(gl[:s0][cov], l0[cov], rtol=2e-5, atol=0)
    o_ref, l_ref = oracle.combine(np.concatenate([a0, a1]), np.concatenate([l0, l1]))
    err = _gpu.row_errors(out.cpu().numpy(), o_ref)
    ok = l_ref > 0
    print(f"  q8 stacked {case} T={T}: max row err = {err[ok].max():.3e}")
    assert (err[ok] <= TOL).all()


def test_stacked_level_refuses_narrow_levels():
    """At most 32 rows per kv sequence: FOLD_E_UNSUPPORTED, nothing launched."""
    wl = make_cascade(seed=3, device="cuda", requests=4, heads=8, kv_heads=1, dim=128,
                      prefix_len=208, suffix_len=16, splits=(2, 1))
    keys = _gpu_q8.encode_cache(wl)
    qq = _gpu_q8.split_query(wl, 0.0)
    lv0 = wl.levels[0]
    k16 = _stack(wl, keys, lv0)
    kv0 = _stacked_view(wl, keys, k16, lv0)
    b, h, d = wl.q.shape
    pa = torch.zeros(2, b, h, d, device="cuda")
    pl = torch.zeros(2, b, h, device="cuda")
    z = torch.zeros(b, h, device="cuda")
    with pytest.raises(F.FoldError) as e:
        F.fold_q8_decode_stacked(kv0, qq, z, 16.0, 2, 0, pa, pl)
    assert e.value.status == F.FOLD_E_UNSUPPORTED


@pytest.mark.parametrize("T", [INF, 16.0])
def test_workload5_full_size(T):
    """The full shared-prefix cascade (64 requests x 8 heads over one 16384-key
    prefix, 1024 own keys each) on a two-plane cache, in the benchmark's launch
    configuration (32 + 8 splits): the stacked prefix level on FP16 keys, the
    suffix on the gated two-plane scan, every row against the oracle."""
    from workloads import make_config
    wl = make_config(5, device="cuda")
    dev = wl.q.device
    keys = _gpu_q8.encode_cache(wl)
    qq = _gpu_q8.split_query(wl, -4.0)
    z = _gpu_q8.estimate(wl, keys, qq)
    levels, _ = _gpu_q8.level_views(wl, keys)
    lv0 = wl.levels[0]
    k16 = _stack(wl, keys, lv0)
    kv0 = _stacked_view(wl, keys, k16, lv0)
    b, h, d = wl.q.shape
    s0, s1 = wl.level_splits
    pa = torch.empty(s0 + s1, b, h, d, device=dev)
    pl = torch.empty(s0 + s1, b, h, device=dev)
    x = torch.full((b, h, lv0.max_seq_len), float("nan"), device=dev)
    pa_d, pl_d = torch.empty_like(pa), torch.empty_like(pl)
    F.fold_q8_decode_stacked(kv0, qq, z, T, s0, 0, pa, pl)
    F.fold_q8_decode_stacked(kv0, qq, z, T, s0, 0, pa_d, pl_d, x_out=x)
    F.fold_q8_decode_split(levels[1], keys, qq, z, T, s1, s0, pa, pl)
    out = torch.empty(b, h, d, device=dev)
    F.fold_combine(pa, pl, out)
    torch.cuda.synchronize()
    assert torch.equal(pa[:s0], pa_d[:s0])
    oi = _adapt.oracle_inputs(wl)
    a_, b_, e_ = (keys.plane_a.cpu().numpy(), keys.plane_b.cpu().numpy(),
                  keys.scale.cpu().numpy().view(np.uint16))
    planes = qq.planes.cpu().numpy()
    qa, qb = planes[:, :, 0], planes[:, :, 1]
    eta = qq.eta.cpu().numpy()
    z64 = z.cpu().double().numpy()
    a0, l0 = q8.decode_level_q8_stacked(q8.stack_queries(qa, qb), eta, q8.stack_keys(a_, b_, e_),
                                        oi["v_bits"], num_kv_heads=1, page_size=wl.page_size,
                                        z=z64, T=T, num_splits=s0, imposed_x=x.cpu().numpy(),
                                        **oi["levels"][0])
    a1, l1 = q8.decode_level_q8(qa, qb, eta, (a_, b_, e_), oi["v_bits"], num_kv_heads=1,
                                page_size=wl.page_size, z=z64, T=T,
                                tau=qq.tau.cpu().numpy(), num_splits=s1, **oi["levels"][1])
    np.testing.assert_allclose(pl.cpu().double().numpy()[:s0], l0, rtol=2e-5)
    o_ref, l_ref = oracle.combine(np.concatenate([a0, a1]), np.concatenate([l0, l1]))
    err = _gpu.row_errors(out.cpu().numpy(), o_ref)
    print(f"  workload 5 two-plane T={T}: {b * h} rows, max row err = {err.max():.3e}")
    assert (err <= TOL).all()
