"""Parity of the block model of BF16 values on the GPU (Section 4, "Depth as a
dial"; Algorithm 1, the tile's virtual row).

Bars: block means and their running update within 1e-5 relative of the FP64
oracle; every scan kernel's cut masses per 16-key chunk within 2e-5 relative
of the oracle's in imposed mode (the kernel's FP32 live decisions); the
virtual rows each slot gains (the block-model slot minus the plain slot)
within 2e-5 of the oracle's sum over tiles of c_it |mu_t| plus a few FP32
units of the slot; L unchanged bit for bit; the combined output within 1e-2
of the row's inf-norm (the decode's bar).
"""

import math

import numpy as np
import pytest
import torch

import oracle
import paper_2609_33410_amd as F
from tests import _adapt, _gpu
from workloads import make_cascade, make_config, make_custom

pytestmark = pytest.mark.gpu
INF = float("inf")
TOL = 1e-2
EPS32 = 2.0 ** -23


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    F.load_library()


def _level_kv(wl, lv):
    return F.kv_view(wl.k, wl.v, lv.seq_lens, num_kv_heads=wl.num_kv_heads,
                     max_seq_len=lv.max_seq_len, block_table=lv.block_table,
                     row_indptr=lv.row_indptr, row_req=lv.row_req,
                     max_reqs_per_seq=lv.max_reqs_per_seq)


def _gpu_block_means(wl, lv, kv):
    bm = torch.full((lv.num_seqs, wl.num_kv_heads, F.block_count(lv.max_seq_len), wl.head_dim),
                    float("nan"), dtype=torch.float32, device=wl.q.device)
    F.fold_value_block_mean(kv, bm)
    return bm


def _oracle_block_means(wl, oi, lv):
    return {(r, g): oracle.block_means(oi["v_bits"], r, g, n, lv["block_table"], wl.page_size)
            for r, n in enumerate(lv["seq_lens"]) for g in range(wl.num_kv_heads)}


@pytest.mark.parametrize("paged,d", [(True, 128), (False, 128), (True, 64)])
def test_block_means(paged, d):
    lens = [0, 1, 17, 64, 65, 333, 1000]
    wl = make_custom(batch=len(lens), heads=8, kv_heads=2, dim=d, lens=lens, paged=paged,
                     seed=3, device="cuda")
    oi = _adapt.oracle_inputs(wl)
    lv = wl.levels[0]
    got = _gpu_block_means(wl, lv, _level_kv(wl, lv))
    torch.cuda.synchronize()
    got = got.cpu().double().numpy()
    want = _oracle_block_means(wl, oi, oi["levels"][0])
    for (r, g), mu in want.items():
        nb = mu.shape[0]
        np.testing.assert_allclose(got[r, g, :nb], mu, rtol=1e-5, atol=1e-6)
        assert not got[r, g, nb:].any()  # blocks past the end are zeros


def test_running_update_of_the_block_means():
    """Block means of the first n - 1 keys, then the n-th key appended (a new
    block when n - 1 is a multiple of 64): the block means of n keys."""
    lens = [5, 65, 129, 300]
    wl = make_custom(batch=4, heads=4, kv_heads=2, dim=64, lens=lens, seed=4, device="cuda")
    lv = wl.levels[0]
    short = (lv.seq_lens - 1).contiguous()
    kv_s = F.kv_view(wl.k, wl.v, short, num_kv_heads=2, max_seq_len=lv.max_seq_len,
                     block_table=lv.block_table)
    bm = _gpu_block_means(wl, lv, kv_s)
    v_new = torch.stack([wl.logical_v[r, :, n - 1] for r, n in enumerate(lens)]).cuda()
    kv = _level_kv(wl, lv)
    F.fold_value_block_mean_append(kv, v_new.contiguous(),
                                   torch.arange(4, dtype=torch.int32, device="cuda"),
                                   short.to(torch.int32), bm)
    torch.cuda.synchronize()
    got = bm.cpu().double().numpy()
    oi = _adapt.oracle_inputs(wl)
    for (r, g), mu in _oracle_block_means(wl, oi, oi["levels"][0]).items():
        np.testing.assert_allclose(got[r, g, :mu.shape[0]], mu, rtol=1e-5, atol=1e-6)


def _chunk_cut_ref(wl, oi, lv, z64, x, T):
    """Oracle cut mass per (row, 16-key chunk) of a level, in imposed mode."""
    q = oracle.bf16_bits_to_f64(oi["q_bits"])
    G = wl.group
    ref = {}
    for seq, n in enumerate(lv["seq_lens"]):
        reqs = [seq] if lv["row_indptr"] is None else \
            list(lv["row_req"][lv["row_indptr"][seq]:lv["row_indptr"][seq + 1]])
        for g in range(wl.num_kv_heads):
            keys = oracle.gather(oi["k_bits"], seq, g, n, lv["block_table"], wl.page_size)
            for r in reqs:
                hs = [g * G + hh for hh in range(G)]
                s = oracle.scores(q[r, hs], keys, wl.sm_scale)
                xx = s - z64[r, hs][:, None]
                live = oracle.live_mask_imposed(x[r, hs, :n], T)
                cw = np.exp2(xx) * ~live
                nch = (n + 15) // 16
                for k, hh in enumerate(hs):
                    ref[(r, hh)] = np.array([cw[k, 16 * c:16 * c + 16].sum() for c in range(nch)])
    return ref


CASES = {
    "mha64": lambda: make_custom(batch=3, heads=4, kv_heads=4, dim=64, lens=[100, 700, 33],
                                 spike_count=4, n_sink=1, seed=8, device="cuda"),
    "mha128_w8": lambda: make_custom(batch=5, heads=2, kv_heads=2, dim=128,
                                     lens=[2100, 1100, 2053, 0, 77], spike_count=6, n_sink=1,
                                     seed=9, device="cuda", splits=3),
    "gqa4": lambda: make_config(2, batch=2, seq_len=1200, seed=2, device="cuda"),
    "gqa8": lambda: make_custom(batch=2, heads=16, kv_heads=2, dim=128, lens=[900, 517],
                                spike_count=5, n_sink=2, seed=10, device="cuda", splits=2),
    "rows16": lambda: make_custom(batch=2, heads=16, kv_heads=1, dim=128, lens=[700, 450],
                                  spike_count=5, n_sink=2, seed=11, device="cuda", splits=2),
    "cascade32": lambda: make_cascade(requests=4, heads=8, kv_heads=1, dim=128, prefix_len=608,
                                      suffix_len=32, splits=(2, 1), seed=6, device="cuda"),
    "stacked40": lambda: make_cascade(requests=5, heads=8, kv_heads=1, dim=128, prefix_len=1488,
                                      suffix_len=48, splits=(3, 2), seed=5, device="cuda"),
    "stacked72_d64": lambda: make_cascade(requests=9, heads=8, kv_heads=1, dim=64,
                                          prefix_len=400, suffix_len=16, splits=(2, 1), seed=7,
                                          device="cuda"),
}


@pytest.mark.parametrize("case", list(CASES))
@pytest.mark.parametrize("T", [INF, 12.0, 4.0])
def test_block_model_every_scan(case, T):
    """Every BF16 scan kernel with the block model: the VALU MHA scan (4 and 8
    waves), the packed GQA scan (4 and 8 rows), the 16- and 32-row matrix-core
    scan and the stacked-row scan (40 and 72 rows)."""
    wl = CASES[case]()
    oi = _adapt.oracle_inputs(wl)
    dev = wl.q.device
    z = _gpu.estimate(wl)
    z64 = z.cpu().double().numpy()
    qv = F.q_view(wl.q)
    b, h, d = wl.q.shape
    splits = list(wl.level_splits)
    tot = sum(splits)
    pa0 = torch.full((tot, b, h, d), float("nan"), device=dev)
    pl0 = torch.full((tot, b, h), float("nan"), device=dev)
    pa1, pl1 = pa0.clone(), pl0.clone()
    pa2, pl2 = pa0.clone(), pl0.clone()
    xs, cuts, means = [], [], []
    off = 0
    for lv, s in zip(wl.levels, splits):
        kv = _level_kv(wl, lv)
        bm = _gpu_block_means(wl, lv, kv)
        x = torch.full((b, h, lv.max_seq_len), float("nan"), device=dev)
        # plain scan (debug exports: the x the kernel compared)
        F.fold_decode_split(kv, qv, wl.sm_scale, z, T, s, off, pa0, pl0, x_out=x)
        # block model, production kernels
        cut = torch.full((b * h * F.chunk_count(lv.max_seq_len),), float("nan"), device=dev)
        F.fold_decode_split_blocks(kv, qv, wl.sm_scale, z, T, s, off, pa1, pl1, bm, cut)
        # block model through the debug kernels (the same sums)
        cut2 = torch.full_like(cut, float("nan"))
        x2 = torch.full_like(x, float("nan"))
        F.fold_decode_split_blocks(kv, qv, wl.sm_scale, z, T, s, off, pa2, pl2, bm, cut2,
                                   x_out=x2)
        xs.append(x)
        cuts.append((cut, cut2))
        means.append(bm)
        off += s
    out = torch.empty(b, h, d, device=dev)
    F.fold_combine(pa1, pl1, out)
    torch.cuda.synchronize()

    # L does not change; the debug kernels give the block-model kernels' slots
    assert not torch.isnan(pl1).any()
    assert torch.equal(pl0, pl1) and torch.equal(pl1, pl2)
    assert torch.allclose(pa1, pa2, rtol=1e-6, atol=0)

    # cut masses per chunk (finite depth)
    for li, (lv, lvo) in enumerate(zip(wl.levels, oi["levels"])):
        x = xs[li].cpu().numpy()
        if math.isinf(T):
            continue
        ref = _chunk_cut_ref(wl, oi, lvo, z64, x, T)
        stride = F.chunk_count(lv.max_seq_len)
        for c in cuts[li]:
            got = c.cpu().double().numpy().reshape(b * h, stride)
            for (r, hh), want in ref.items():
                g_row = got[r * h + hh, :want.size]
                pos = want > 0
                assert np.allclose(g_row[pos], want[pos], rtol=2e-5, atol=0), (r, hh)
                assert np.all(g_row[~pos] <= 1e-30), (r, hh)

    # the virtual rows each slot gains
    pa_ref, pa_plain, pa_abs, pl_ref = [], [], [], []
    for li, (lvo, s) in enumerate(zip(oi["levels"], splits)):
        ob = _oracle_block_means(wl, oi, lvo)
        gb = means[li].cpu().double().numpy()
        for (r, g), mu in ob.items():
            np.testing.assert_allclose(gb[r, g, :mu.shape[0]], mu, rtol=1e-5, atol=1e-6)
        kw = dict(num_kv_heads=wl.num_kv_heads, page_size=wl.page_size, sm_scale=wl.sm_scale,
                  z=z64, T=T, num_splits=s, imposed_x=xs[li].cpu().numpy(), **lvo)
        a_b, l_b = oracle.decode_level(oi["q_bits"], oi["k_bits"], oi["v_bits"],
                                       block_mean=ob, **kw)
        a_p, _ = oracle.decode_level(oi["q_bits"], oi["k_bits"], oi["v_bits"], **kw)
        a_abs, _ = oracle.decode_level(oi["q_bits"], oi["k_bits"], oi["v_bits"],
                                       block_mean={k: np.abs(v) for k, v in ob.items()}, **kw)
        pa_ref.append(a_b), pa_plain.append(a_p), pa_abs.append(a_abs - a_p), pl_ref.append(l_b)
    pa_ref, pa_plain = np.concatenate(pa_ref), np.concatenate(pa_plain)
    scale, pl_ref = np.concatenate(pa_abs), np.concatenate(pl_ref)
    covered = pl_ref > 0
    g1 = pa1.cpu().double().numpy()
    g0 = pa0.cpu().double().numpy()
    dv_gpu = (g1 - g0)[covered]
    dv_ref = (pa_ref - pa_plain)[covered]
    tol = 2e-5 * scale[covered] + 8 * EPS32 * (np.abs(g1[covered]) + np.abs(g0[covered]))
    worst = float((np.abs(dv_gpu - dv_ref) / np.maximum(tol, 1e-300)).max()) if dv_ref.size else 0
    if not math.isinf(T):
        assert scale.max() > 0
    assert (np.abs(dv_gpu - dv_ref) <= tol).all(), worst

    # the combined output
    o_ref, l_ref = oracle.combine(pa_ref, pl_ref)
    ok = l_ref > 0
    err = _gpu.row_errors(out.cpu().numpy(), o_ref)
    print(f"  blocks {case} T={T}: virtual-row err / tol = {worst:.3f}, "
          f"max row err = {err[ok].max():.3e}")
    assert (err[ok] <= TOL).all()


@pytest.mark.parametrize("case", ["mha64", "gqa4", "stacked40"])
def test_blockwise_constant_values_make_the_block_model_exact(case):
    """Value rows constant within every 64-key block: the block model's output
    at a finite depth equals the dense output (to FP32 rounding)."""
    wl = CASES[case]()
    gen = torch.Generator(device="cpu").manual_seed(12)
    # one value per (logical 64-key block) written through the block tables
    b, h, d = wl.q.shape
    if wl.page_size:
        # pages hold 16 keys: logical block t of a sequence covers its pages 4t .. 4t+3
        per = torch.randn(wl.v.shape[0], wl.num_kv_heads, d, generator=gen).to(torch.bfloat16)
        v = torch.empty_like(wl.v)
        for lv in wl.levels:
            bt = lv.block_table.cpu()
            for sq in range(lv.num_seqs):
                npg = (lv.seq_lens_host[sq] + 15) // 16
                for p in range(npg):
                    phys = int(bt[sq, p])
                    anchor = int(bt[sq, (p // 4) * 4])
                    v[phys] = per[anchor].to(v.device)[:, None, :].expand(-1, 16, -1)
        wl.v = v.contiguous()
    else:
        n_max = wl.v.shape[2]
        per = torch.randn(wl.v.shape[0], wl.v.shape[1], (n_max + 63) // 64, d, generator=gen)
        wl.v = per.to(torch.bfloat16).repeat_interleave(64, dim=2)[:, :, :n_max].contiguous() \
            .to(wl.q.device)
    z = _gpu.estimate(wl)
    qv = F.q_view(wl.q)
    splits = list(wl.level_splits)
    outs = {}
    for T in (INF, 4.0):
        pa = torch.empty(sum(splits), b, h, d, device=wl.q.device)
        pl = torch.empty(sum(splits), b, h, device=wl.q.device)
        off = 0
        for lv, s in zip(wl.levels, splits):
            kv = _level_kv(wl, lv)
            bm = _gpu_block_means(wl, lv, kv)
            cut = torch.empty(b * h * F.chunk_count(lv.max_seq_len), device=wl.q.device)
            F.fold_decode_split_blocks(kv, qv, wl.sm_scale, z, T, s, off, pa, pl, bm, cut)
            off += s
        o = torch.empty(b, h, d, device=wl.q.device)
        F.fold_combine(pa, pl, o)
        outs[T] = o
    torch.cuda.synchronize()
    dense, model = outs[INF].double(), outs[4.0].double()
    scale = dense.abs().amax(dim=-1).clamp_min(1e-30)
    err = float(((model - dense).abs().amax(dim=-1) / scale).max())
    print(f"  blockwise-constant {case}: max row err vs dense = {err:.3e}")
    assert err < 1e-4


@pytest.mark.parametrize("cfg,chunks", [(3, [(0, 0), (7, 5)]), (4, [(0, 3), (2, 17)])])
def test_block_model_full_size_sampled(cfg, chunks):
    """Full-size workloads 3 (GQA, 32K keys, 16 splits) and 4 (MHA, 64K-128K
    ragged, 32 splits) at T = 16 with the block model, in the launch
    configuration the benchmark times: the sampled (kv sequence, kv head)
    chunks' rows against the oracle (block means of those chunks, the
    kernel's FP32 live decisions)."""
    wl = make_config(cfg, device="cuda")
    dev = wl.q.device
    T = 16.0
    lv = wl.levels[0]
    kv = _level_kv(wl, lv)
    qv = F.q_view(wl.q)
    z = _gpu.estimate(wl)
    b, h, d = wl.q.shape
    s = wl.level_splits[0]
    bm = _gpu_block_means(wl, lv, kv)
    cut = torch.empty(b * h * F.chunk_count(lv.max_seq_len), device=dev)
    pa = torch.empty(s, b, h, d, device=dev)
    pl = torch.empty(s, b, h, device=dev)
    F.fold_decode_split_blocks(kv, qv, wl.sm_scale, z, T, s, 0, pa, pl, bm, cut)
    out = torch.empty(b, h, d, device=dev)
    F.fold_combine(pa, pl, out)
    x = torch.full((b, h, lv.max_seq_len), float("nan"), device=dev)
    pa_d, pl_d = torch.empty_like(pa), torch.empty_like(pl)
    F.fold_decode_split_blocks(kv, qv, wl.sm_scale, z, T, s, 0, pa_d, pl_d, bm, cut, x_out=x)
    torch.cuda.synchronize()
    oi = _adapt.oracle_inputs(wl)
    lvo = oi["levels"][0]
    z64 = z.cpu().double().numpy()
    ob = {(r, g): oracle.block_means(oi["v_bits"], r, g, lvo["seq_lens"][r], lvo["block_table"],
                                     wl.page_size) for r, g in chunks}
    gb = bm.cpu().double().numpy()
    for (r, g), mu in ob.items():
        np.testing.assert_allclose(gb[r, g, :mu.shape[0]], mu, rtol=1e-5, atol=1e-6)
    a_r, l_r = oracle.decode_level(oi["q_bits"], oi["k_bits"], oi["v_bits"],
                                   num_kv_heads=wl.num_kv_heads, page_size=wl.page_size,
                                   sm_scale=wl.sm_scale, z=z64, T=T, num_splits=s,
                                   imposed_x=x.cpu().numpy(), chunks=chunks, block_mean=ob,
                                   **lvo)
    o_ref, _ = oracle.combine(a_r, l_r)
    G = wl.group
    rows = [(r, g * G + hh) for r, g in chunks for hh in range(G)]
    ri = np.array([r for r, _ in rows])
    hi = np.array([hh for _, hh in rows])
    err = _gpu.row_errors(out.cpu().numpy()[ri, hi], o_ref[ri, hi])
    gpa = pa.cpu().double().numpy()[:, ri, hi]
    dense_rel = np.abs(gpa - a_r[:, ri, hi]).max() / np.abs(a_r[:, ri, hi]).max()
    print(f"  {wl.name} T=16 block model: sampled rows {len(rows)}, max row err = {err.max():.3e},"
          f" slot A max rel = {dense_rel:.3e}")
    assert (err <= TOL).all()
    np.testing.assert_allclose(pl.cpu().double().numpy()[:, ri, hi], l_r[:, ri, hi], rtol=2e-5)
