"""Parity of the cut-key value model on the GPU (Section 4, "Depth as a dial").

Bars: request means and their running update within 1e-5 relative of the
FP64 oracle; every scan kernel's cut masses within 2e-5 relative of the
oracle's in imposed mode (the kernel's FP32 decisions), zero at T = inf; the
combined output with the model within 1e-2 of the row's inf-norm.
"""

import math

import numpy as np
import pytest
import torch

import oracle
import paper_2609_33410_amd as F
from oracle import q8_oracle as q8
from tests import _adapt, _gpu, _gpu_q8
from workloads import host_bits, make_cascade, make_config, make_custom

pytestmark = pytest.mark.gpu
INF = float("inf")
TOL = 1e-2


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    F.load_library()


def _oracle_means(wl, oi):
    fl = oi["flat"]
    return np.stack([np.stack([oracle.value_mean(oi["v_bits"], r, g, n, fl["block_table"],
                                                 wl.page_size)
                               for g in range(wl.num_kv_heads)])
                     for r, n in enumerate(fl["seq_lens"])])


def _gpu_means(wl):
    fl = wl.flat
    kv = F.kv_view(wl.k, wl.v, fl.seq_lens, num_kv_heads=wl.num_kv_heads,
                   max_seq_len=fl.max_seq_len, block_table=fl.block_table)
    mean = torch.full((fl.num_seqs, wl.num_kv_heads, wl.head_dim), float("nan"),
                      dtype=torch.float32, device=wl.q.device)
    F.fold_value_mean(kv, mean)
    return mean


@pytest.mark.parametrize("paged", [True, False])
def test_request_means(paged):
    lens = [0, 1, 17, 64, 333, 1000]
    wl = make_custom(batch=len(lens), heads=8, kv_heads=2, dim=128, lens=lens, paged=paged,
                     seed=3, device="cuda")
    oi = _adapt.oracle_inputs(wl)
    got = _gpu_means(wl).cpu().double().numpy()
    want = _oracle_means(wl, oi)
    assert np.array_equal(got[0], np.zeros_like(got[0]))
    np.testing.assert_allclose(got, want, rtol=1e-5, atol=1e-6)


def test_running_update_of_the_means():
    """Means of the first n - 1 keys, then the n-th key appended: the mean of n."""
    lens = [5, 40, 300]
    wl = make_custom(batch=3, heads=4, kv_heads=2, dim=64, lens=lens, seed=4, device="cuda")
    fl = wl.flat
    short = (fl.seq_lens - 1).contiguous()
    kv_s = F.kv_view(wl.k, wl.v, short, num_kv_heads=2, max_seq_len=fl.max_seq_len,
                     block_table=fl.block_table)
    mean = torch.empty(3, 2, 64, dtype=torch.float32, device="cuda")
    F.fold_value_mean(kv_s, mean)
    # the appended tokens' value rows, read from the logical cache
    v_new = torch.stack([wl.logical_v[r, :, n - 1] for r, n in enumerate(lens)]).cuda()
    kv = F.kv_view(wl.k, wl.v, fl.seq_lens, num_kv_heads=2, max_seq_len=fl.max_seq_len,
                   block_table=fl.block_table)
    F.fold_value_mean_append(kv, v_new.contiguous(), torch.arange(3, dtype=torch.int32).cuda(),
                             short.to(torch.int32), mean)
    torch.cuda.synchronize()
    oi = _adapt.oracle_inputs(wl)
    np.testing.assert_allclose(mean.cpu().double().numpy(), _oracle_means(wl, oi), rtol=1e-5,
                               atol=1e-6)


def _run_with_cut(wl, T, splits=None):
    """BF16 path with cut masses; returns host tensors and the exported x."""
    dev = wl.q.device
    splits = list(splits or wl.level_splits)
    levels, flat = _gpu.kv_views(wl)
    qv = F.q_view(wl.q)
    z = _gpu.estimate(wl)
    b, h, d = wl.q.shape
    tot = sum(splits)
    pa = torch.empty(tot, b, h, d, device=dev)
    pl = torch.empty(tot, b, h, device=dev)
    pc = torch.zeros(tot, b, h, device=dev)  # rows a level does not cover keep 0
    xs = []
    off = 0
    for lv, kv, s in zip(wl.levels, levels, splits):
        x = torch.full((b, h, lv.max_seq_len), float("nan"), device=dev)
        F.fold_decode_split(kv, qv, wl.sm_scale, z, T, s, off, pa, pl, x_out=x, part_Lcut=pc)
        xs.append(x)
        off += s
    mean = _gpu_means(wl)
    out = torch.empty(b, h, d, device=dev)
    F.fold_combine(pa, pl, out, part_Lcut=pc, mean=mean)
    torch.cuda.synchronize()
    return {"z": z.cpu().double().numpy(), "pa": pa.cpu(), "pl": pl.cpu(), "pc": pc.cpu(),
            "x": [x.cpu().numpy() for x in xs], "out": out.cpu().numpy(),
            "mean": mean.cpu().double().numpy(), "splits": splits}


def _oracle_with_cut(wl, oi, res, T):
    pa, pl, pc = [], [], []
    for li, (lv, s) in enumerate(zip(oi["levels"], res["splits"])):
        a, l, c = oracle.decode_level(oi["q_bits"], oi["k_bits"], oi["v_bits"],
                                      num_kv_heads=wl.num_kv_heads, page_size=wl.page_size,
                                      sm_scale=wl.sm_scale, z=res["z"], T=T, num_splits=s,
                                      imposed_x=res["x"][li], with_cut=True, **lv)
        pa.append(a), pl.append(l), pc.append(c)
    pa, pl, pc = np.concatenate(pa), np.concatenate(pl), np.concatenate(pc)
    o, l = oracle.combine(pa, pl, pc, _oracle_means(wl, oi), wl.num_kv_heads)
    return o, l, pc


@pytest.mark.parametrize("case", ["mha", "gqa", "stacked", "cascade32"])
@pytest.mark.parametrize("T", [INF, 12.0, 4.0])
def test_cut_masses_and_model_output(case, T):
    """Every BF16 scan kernel: the VALU MHA scan, the GQA matrix-core scan, the
    stacked-row scan (40 rows on the prefix) and 32 stacked rows (GQA scan)."""
    if case == "mha":
        wl = make_custom(batch=3, heads=4, kv_heads=4, dim=64, lens=[100, 700, 33],
                         spike_count=4, n_sink=1, seed=8, device="cuda")
    elif case == "gqa":
        wl = make_config(2, batch=2, seq_len=1200, seed=2, device="cuda")
    elif case == "stacked":
        wl = make_cascade(requests=5, heads=8, kv_heads=1, dim=128, prefix_len=1488,
                          suffix_len=48, splits=(3, 2), seed=5, device="cuda")
    else:
        wl = make_cascade(requests=4, heads=8, kv_heads=1, dim=128, prefix_len=608,
                          suffix_len=32, splits=(2, 1), seed=6, device="cuda")
    oi = _adapt.oracle_inputs(wl)
    res = _run_with_cut(wl, T)
    o_ref, l_ref, pc_ref = _oracle_with_cut(wl, oi, res, T)
    gc = res["pc"].double().numpy()
    if math.isinf(T):
        assert not gc.any()
    cov = pc_ref > 0
    assert np.allclose(gc[cov], pc_ref[cov], rtol=2e-5, atol=0)
    assert np.all(gc[~cov] <= 1e-30)
    ok = l_ref > 0
    err = _gpu.row_errors(res["out"], o_ref)
    print(f"  model {case} T={T}: max row err = {err[ok].max():.3e}, cut mass share = "
          f"{gc.sum() / max(res['pl'].double().numpy().sum(), 1e-300):.3e}")
    assert (err[ok] <= TOL).all()


def test_model_is_exact_for_constant_values():
    """All value rows equal c: with the model the output is c at any depth."""
    wl = make_config(2, batch=2, seq_len=900, seed=1, device="cuda")
    c = torch.linspace(-1, 1, wl.head_dim, device="cuda").to(torch.bfloat16)
    wl.v = c.expand_as(wl.v).contiguous()
    for T in (2.0, 8.0):
        res = _run_with_cut(wl, T)
        assert np.abs(res["out"] - c.float().cpu().numpy()).max() < 1e-5


@pytest.mark.parametrize("T", [INF, 8.0])
def test_two_plane_cut_masses(T):
    wl = make_config(2, batch=2, seq_len=1000, device="cuda")
    oi = _adapt.oracle_inputs(wl)
    keys = _gpu_q8.encode_cache(wl)
    qq = _gpu_q8.split_query(wl, 0.0)
    levels, flat = _gpu_q8.level_views(wl, keys)
    z = _gpu_q8.estimate(wl, keys, qq)
    b, h, d = wl.q.shape
    pa = torch.empty(3, b, h, d, device="cuda")
    pl = torch.empty(3, b, h, device="cuda")
    pc = torch.empty(3, b, h, device="cuda")
    xc = torch.full((b, h, 1000), float("nan"), device="cuda")
    x = torch.full((b, h, 1000), float("nan"), device="cuda")
    F.fold_q8_decode_split(levels[0], keys, qq, z, T, 3, 0, pa, pl, xc_out=xc, x_out=x,
                           part_Lcut=pc)
    torch.cuda.synchronize()
    planes = q8.split_keys(host_bits(wl.k))
    qa, qb, eta = q8.split_queries(host_bits(wl.q), wl.sm_scale)
    tau = np.array([q8.refine_tau(n, 0.0) for n in wl.flat.seq_lens_host], dtype=np.float32)
    _, pl_ref, pc_ref = q8.decode_level_q8(qa, qb, eta, planes, oi["v_bits"],
                                           num_kv_heads=wl.num_kv_heads, page_size=wl.page_size,
                                           z=z.cpu().double().numpy(), T=T, tau=tau,
                                           num_splits=3, imposed=(xc.cpu().numpy(),
                                                                  x.cpu().numpy()),
                                           with_cut=True, **oi["levels"][0])
    gc = pc.cpu().double().numpy()
    if math.isinf(T):
        assert not gc.any()
    cov = pc_ref > 0
    assert np.allclose(gc[cov], pc_ref[cov], rtol=2e-5, atol=0)
